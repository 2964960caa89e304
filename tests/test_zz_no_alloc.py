"""The entry point that allocates nothing (avsg_step_static, for callers that
cannot allocate) against avsg_step on a handle: the same slots, miss counts
and buffer bytes after every step, over two call sequences in a row, the
second with a smaller configuration, and across the transfers it supports."""
import numpy as np
import pytest

import workload as W
from harness import GpuSide, HostRows, compare_step, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2609_37538_amd import avsg as A
    A.load()            # fails loudly when the HIP library is missing
    W.build(force=False)


def _run_pair(spec, gather_mode, match_mode=0):
    """Step spec through a handle and through avsg_step_static (cold start at
    step 0, continuing calls after it) on the same inputs and host rows."""
    import torch
    from paper_2609_37538_amd import avsg as A
    wl = W.Workload(spec)
    host = HostRows(wl)
    ref = GpuSide(wl, host, gather_mode=gather_mode, match_mode=match_mode)
    cfg = ref.cfg
    B, K, n_q, S = spec.batch, spec.topk, spec.n_q, spec.slots
    dev = torch.device("cuda")
    bufs = [torch.zeros((B, S, rb), dtype=torch.uint8, device=dev) for rb in spec.row_bytes]
    buf_ptrs = [bufs[s][r].data_ptr() for s in range(len(bufs)) for r in range(B)]
    slots = torch.empty((B, n_q, K), dtype=torch.int32, device=dev)
    counts = torch.empty((B, n_q), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    log(f"[no-alloc] {spec.name}: B={B} K={K} n_q={n_q} S={S} gather={gather_mode} match={match_mode}")
    try:
        for t in range(spec.steps):
            X = wl.topk(t)
            N = wl.verified_len(t) if spec.speculative else None
            W.refresh_speculative(wl, t, host.stream_ptrs())
            O_ref, n_ref = ref.step(X, N)
            Xd = torch.from_numpy(X).to(dev)
            Nd = None if N is None else torch.from_numpy(N).to(dev)
            A.avsg_step_static(cfg, host.ptrs, wl.ctx, buf_ptrs, Xd.data_ptr(),
                               None if Nd is None else Nd.data_ptr(), slots.data_ptr(), counts.data_ptr(),
                               cold_start=(t == 0), stream=stream)
            torch.cuda.synchronize()
            compare_step(t, O_ref, n_ref, slots.cpu().numpy(), counts.cpu().numpy())
            if gather_mode != A.AVSG_GATHER_NONE and (t % 4 == 0 or t == spec.steps - 1):
                want = ref.buffers()
                for s in range(len(bufs)):
                    assert np.array_equal(bufs[s].cpu().numpy(), want[s]), f"step {t} stream {s}: buffers differ"
    finally:
        ref.close()
        host.free()


def test_static_step_two_calls_second_smaller():
    """A resident-reuse batch with two query tokens and two row streams, then a
    smaller single-token batch with the paper's Stage Two: each sequence
    starts cold and continues on the tables the previous call left."""
    from paper_2609_37538_amd import avsg as A
    big = W.custom_spec(name="static_big", batch=6, topk=512, slots=2048, n_q=2, steps=10, ctx=20000,
                        row_bytes=(1152, 132), retention=0.85)
    small = W.custom_spec(name="static_small", batch=3, topk=256, slots=1024, n_q=1, steps=6, ctx=5000)
    _run_pair(big, A.AVSG_GATHER_RESIDENT)
    _run_pair(small, A.AVSG_GATHER_BALANCED)


@pytest.mark.parametrize("gather_mode,match_mode", [(1, 0), (4, 0), (3, 0), (0, 1), (1, 1)],
                         ids=["request_level", "position_level", "match_only", "dualptr", "dualptr_request"])
def test_static_step_other_transfers(gather_mode, match_mode):
    spec = W.custom_spec(name=f"static_{gather_mode}_{match_mode}", batch=4,
                         topk=256, slots=256 if match_mode else 1024, n_q=1, steps=8, ctx=6000)
    _run_pair(spec, gather_mode, match_mode)


def test_static_step_speculative_rows():
    """Verified lengths and rewritten draft rows: invalidation runs in the
    static step as on a handle."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name="static_spec", batch=2, topk=256, slots=2048, n_q=3, steps=12, ctx=4096,
                         mode="zipf_window", window=64, retention=0.8)
    _run_pair(spec, A.AVSG_GATHER_RESIDENT)


def test_static_step_refusals():
    """Host-side refusals: a layout beyond the static array, validate mode or
    a transfer the static step does not run, and a continuing call after a
    call with another configuration."""
    import torch
    from paper_2609_37538_amd import avsg as A
    fake = [4096 * (i + 1) for i in range(2 * 512)]

    def status(cfg, B, cold=True):
        try:
            A.avsg_step_static(cfg, fake[:cfg.n_streams * B], [1 << 20] * B, fake[:cfg.n_streams * B],
                               4096, None, 4096, 4096, cold_start=cold,
                               stream=torch.cuda.current_stream().cuda_stream)
        except A.AvsgError as e:
            return e.status
        return A.AVSG_OK

    huge = A.make_config(256, 2048, 2, 8192, row_bytes=(1152, 132), gather_mode=A.AVSG_GATHER_RESIDENT)
    assert A.avsg_workspace_bytes(huge) > (32 << 20)
    assert status(huge, 256) == A.AVSG_E_CAPACITY
    assert status(A.make_config(2, 64, 1, 256, validate=1), 2) == A.AVSG_E_UNSUPPORTED
    assert status(A.make_config(2, 64, 1, 256, gather_mode=A.AVSG_GATHER_EARLY), 2) == A.AVSG_E_UNSUPPORTED
    # the last successful call (if any) had another configuration
    assert status(A.make_config(2, 64, 1, 512, retry=2, max_life=5), 2, cold=False) == A.AVSG_E_INVAL


@pytest.mark.parametrize("gather_mode", [6, 0], ids=["resident", "balanced"])
def test_static_step_graph_replays(gather_mode):
    """A continuing avsg_step_static call captured into a HIP graph (the caller
    it exists for) and replayed once per decode step, the next selections
    copied into the captured input between replays: after every replay the
    slots, counts and buffers equal a handle stepped eagerly."""
    import torch
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"static_graph_{gather_mode}", batch=4, topk=256, slots=1024, n_q=2, steps=10,
                         ctx=6000, row_bytes=(1152, 132), retention=0.8)
    wl = W.Workload(spec)
    host = HostRows(wl)
    ref = GpuSide(wl, host, gather_mode=gather_mode)
    cfg = ref.cfg
    B, K, n_q, S = spec.batch, spec.topk, spec.n_q, spec.slots
    dev = torch.device("cuda")
    bufs = [torch.zeros((B, S, rb), dtype=torch.uint8, device=dev) for rb in spec.row_bytes]
    buf_ptrs = [bufs[s][r].data_ptr() for s in range(len(bufs)) for r in range(B)]
    slots = torch.empty((B, n_q, K), dtype=torch.int32, device=dev)
    counts = torch.empty((B, n_q), dtype=torch.int32, device=dev)
    X_in = torch.zeros((B, n_q, K), dtype=torch.int32, device=dev)
    side = torch.cuda.Stream()
    log(f"[no-alloc graph] {spec.name}: B={B} K={K} n_q={n_q} S={S} gather={gather_mode}")

    def static_step(cold):
        A.avsg_step_static(cfg, host.ptrs, wl.ctx, buf_ptrs, X_in.data_ptr(), None, slots.data_ptr(),
                           counts.data_ptr(), cold_start=cold, stream=side.cuda_stream)

    def check(t, X):
        O_ref, n_ref = ref.step(X, None)
        torch.cuda.synchronize()
        compare_step(t, O_ref, n_ref, slots.cpu().numpy(), counts.cpu().numpy())
        want = ref.buffers()
        for s in range(len(bufs)):
            assert np.array_equal(bufs[s].cpu().numpy(), want[s]), f"step {t} stream {s}: buffers differ"

    g = torch.cuda.CUDAGraph()
    try:
        # step 0 eagerly, from a cold start
        X = wl.topk(0)
        X_in.copy_(torch.from_numpy(np.ascontiguousarray(X, dtype=np.int32)).to(dev))
        torch.cuda.synchronize()
        static_step(True)
        check(0, X)
        with torch.cuda.graph(g, stream=side):
            static_step(False)
        torch.cuda.synchronize()
        for t in range(1, spec.steps):
            log(f"[no-alloc graph] replay {t}")
            X = wl.topk(t)
            X_in.copy_(torch.from_numpy(np.ascontiguousarray(X, dtype=np.int32)).to(dev))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            check(t, X)
    finally:
        del g
        ref.close()
        host.free()
