"""GPU parity: the HIP operator (through the C ABI) against the CPU oracle on the
same seeded inputs and the same pinned host rows, bit-exact: slot map, miss
counts, transfer lists, table state (c_j and q_j), counters and buffer bytes.
"""
import json
import os

import numpy as np
import pytest

import oracle as ORC
import workload as W
from harness import (GpuSide, HostRows, OracleSide, compare_step, content_check, log, run_parity,
                     run_parity_modes)

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2609_37538_amd import avsg as A
    A.load()            # fails loudly when the HIP library is missing
    W.build(force=False)
    ORC.build(force=False)


def test_hand_trace_on_gpu():
    """The hand-traced S = 8 example through the GPU path."""
    from paper_2609_37538_amd import avsg as A
    import torch
    g = json.load(open(os.path.join(GOLDEN, "hand_trace_s8.json")))
    c = g["config"]
    log("[gpu] hand trace S=8")
    host = A.HostRegion(64 * 16)
    host.view()[:] = np.arange(64 * 16, dtype=np.uint32).astype(np.uint8)
    cfg = A.make_config(1, c["topk"], c["n_q"], c["slots"], retry=c["retry"], max_life=c["max_life"],
                        a1=c["a1"], a2=c["a2"], row_bytes=(16,))
    op = A.Operator(cfg, [host.ptr], [64])
    try:
        for k, s in enumerate(g["steps"]):
            X = torch.tensor([s["X"]], dtype=torch.int32, device="cuda")
            N = torch.tensor([s["N"]], dtype=torch.int64, device="cuda")
            O, n = op.step(X, N)
            torch.cuda.synchronize()
            assert O[0].cpu().tolist() == s["O"], f"step {k}"
            assert n[0].cpu().tolist() == s["n"], f"step {k}"
            mx, mo = op.export_misses(0)
            assert mx.tolist() == s["miss_x"] and mo.tolist() == s["miss_o"]
        cc, q = op.export_state(0)
        assert cc.tolist() == g["final_c"]
        life = ((q >> 24).astype(np.uint8)).astype(np.int8).tolist()
        assert life == g["final_life"]
        for j, (b, fp, slot) in enumerate(g["final_buckets"]):
            w = int(q[j]) & 0xFFFFFF
            assert (w >> 23, (w >> 3) & 0xFFFFF, w & 7) == (b, fp, slot), f"bucket {j}"
        st = op.stats()
        for k, v in g["counters"].items():
            assert st[k] == v, k
        buf = op.buffers[0].cpu().numpy()[0]
        rows = host.view().reshape(64, 16)
        for s in g["steps"][-1:]:
            for gi, row in enumerate(s["X"]):
                for i, x in enumerate(row):
                    assert np.array_equal(buf[s["O"][gi][i]], rows[x])
    finally:
        op.close()
        host.free()


def test_parity_tiny():
    """1 request, context 8192, K = 256, S = 1024: every step, every table,
    with the balanced (S3, Eq. 6), request-level (S1, Eq. 13), position-level
    (S2, Eq. 14) and resident-reuse transfers side by side."""
    run_parity_modes(W.get_spec("tiny"), (0, 1, 4, 6), table_every=1, buffers_every=8,
                     miss_list_requests=1)


EDGE_CASES = [
    # name, kwargs of workload.custom_spec
    ("ragged_k", dict(batch=3, topk=100, slots=256, n_q=1, steps=20, ctx=3000)),
    ("k_1000_mtp3", dict(batch=2, topk=1000, slots=4096, n_q=3, steps=12, ctx=50000)),
    ("capacity_exact", dict(batch=2, topk=512, slots=2048, n_q=4, steps=16, ctx=20000)),
    ("k_one", dict(batch=5, topk=1, slots=2, n_q=1, steps=40, ctx=6)),
    ("k_3000", dict(batch=2, topk=3000, slots=8192, n_q=2, steps=8, ctx=100000)),
    ("k_4096_max", dict(batch=1, topk=4096, slots=8192, n_q=2, steps=6, ctx=200000)),
    ("s_16384_max", dict(batch=2, topk=1024, slots=16384, n_q=3, steps=8, ctx=300000)),
    ("mtp_8_tokens", dict(batch=2, topk=128, slots=1024, n_q=8, steps=10, ctx=5000)),
    ("tiny_context", dict(batch=4, topk=64, slots=128, n_q=2, steps=30, ctx=200, retention=0.5)),
    ("all_hits", dict(batch=2, topk=256, slots=1024, n_q=2, steps=10, ctx=256, retention=1.0, overlap=1.0)),
    ("row_132_only", dict(batch=2, topk=128, slots=512, n_q=1, steps=10, ctx=4000, row_bytes=(132,))),
    ("two_streams_odd", dict(batch=3, topk=200, slots=512, n_q=2, steps=10, ctx=9000, row_bytes=(1152, 132))),
    ("spec_window", dict(batch=2, topk=256, slots=2048, n_q=3, steps=20, ctx=4096, mode="zipf_window",
                         window=64, retention=0.8)),
    ("batch_200", dict(batch=200, topk=128, slots=256, n_q=2, steps=6, ctx=2000)),
    ("batch_1024_max", dict(batch=1024, topk=16, slots=64, n_q=2, steps=6, ctx=400)),
    # four-wave workgroups (S <= 1024, K <= 512): two indices per thread, a ragged K
    ("four_waves_two_per_thread", dict(batch=3, topk=512, slots=1024, n_q=2, steps=12, ctx=8000)),
    ("four_waves_ragged", dict(batch=2, topk=300, slots=512, n_q=1, steps=12, ctx=3000)),
]


@pytest.mark.parametrize("name,kw", EDGE_CASES, ids=[e[0] for e in EDGE_CASES])
def test_parity_edge_cases(name, kw):
    spec = W.custom_spec(name=name, **kw)
    run_parity(spec, table_every=1, buffers_every=1, miss_list_requests=3)


@pytest.mark.parametrize("retry,max_life", [(0, 1), (1, 2), (7, 4), (3, 127)])
def test_parity_parameters(retry, max_life):
    """Probe budgets and lifetimes at and near their limits."""
    spec = W.custom_spec(name=f"params_{retry}_{max_life}", batch=3, topk=256, slots=1024, n_q=2,
                         steps=24, ctx=6000, retention=0.7)
    run_parity(spec, table_every=4, buffers_every=8, retry=retry, max_life=max_life)


@pytest.mark.parametrize("mode", [1, 2, 4, 5, 6],
                         ids=["request_level", "copy_engine", "position_level", "pipelined", "resident"])
def test_gather_modes_match_balanced(mode):
    """Request-level (S1), position-level (S2), copy-engine, pipelined and
    resident-reuse transfers leave the same bytes as the balanced miss-list
    transfer (S3)."""
    spec = W.custom_spec(name=f"mode{mode}", batch=6, topk=512, slots=2048, n_q=2, steps=12,
                         ctx=30000, row_bytes=(1152, 132))
    run_parity(spec, table_every=0, buffers_every=4, gather_mode=mode)


@pytest.mark.parametrize("workers", [1, 3, 7, 9, 13, 1000])
def test_range_transfers_worker_counts(workers):
    """S3 (Eq. 6) and S2 (Eq. 14) with grids whose size is not a multiple of
    the eight XCDs, from one workgroup to more workgroups than rows: the
    workgroup-to-worker order that gives consecutive workers to one XCD must
    still hand every worker exactly one range, so every buffer byte equals the
    oracle's.  Three tokens, so rows missed by several tokens of a step
    (served from L2) are among them."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"range_workers_{workers}", batch=3, topk=256, slots=1024, n_q=3, steps=10,
                         ctx=3000, retention=0.8, row_bytes=(1152, 132))
    run_parity_modes(spec, (A.AVSG_GATHER_BALANCED, A.AVSG_GATHER_POSITION), table_every=0, buffers_every=1,
                     miss_list_requests=3, retry=0, gather_workers=workers)


@pytest.mark.parametrize("batch,n_q", [(2, 1), (2, 2)], ids=["s3_side", "resident_side"])
def test_auto_transfer_parity(batch, n_q):
    """AVSG_GATHER_AUTO on both sides of its threshold (4096 and 8192 lookups
    per step): slots, tables, counters and buffers equal the oracle's."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"auto_{batch}_{n_q}", batch=batch, topk=2048, slots=8192, n_q=n_q, steps=10,
                         ctx=60000, row_bytes=(1152, 132))
    cfg = A.make_config(batch, 2048, n_q, 8192, row_bytes=(1152, 132), gather_mode=A.AVSG_GATHER_AUTO)
    want = A.AVSG_GATHER_RESIDENT if batch * n_q * 2048 >= 8192 else A.AVSG_GATHER_BALANCED
    assert A.avsg_resolve_config(cfg).gather_mode == want
    ref, got = run_parity(spec, table_every=2, buffers_every=2, gather_mode=A.AVSG_GATHER_AUTO)
    assert (got["resident_rows"] + got["duplicate_rows"] > 0) == (want == A.AVSG_GATHER_RESIDENT)


def test_lds_capacity_error():
    """A table larger than one workgroup's LDS is refused at create time."""
    from paper_2609_37538_amd import avsg as A
    host = A.HostRegion(1 << 20)
    cfg = A.make_config(1, 2048, 1, 32768, row_bytes=(16,))
    try:
        with pytest.raises(A.AvsgError) as e:
            A.Operator(cfg, [host.ptr], [65536])
        assert e.value.status == A.AVSG_E_CAPACITY
    finally:
        host.free()


def test_match_only_leaves_buffers():
    spec = W.custom_spec(name="match_only", batch=2, topk=128, slots=512, n_q=1, steps=5, ctx=2000)
    wl = W.Workload(spec)
    host = HostRows(wl)
    orc = OracleSide(wl, host, images=False)
    gpu = GpuSide(wl, host, gather_mode=3)
    try:
        for t in range(spec.steps):
            X, N = wl.topk(t), wl.verified_len(t)
            O_ref, n_ref = orc.step(X, N)
            O_gpu, n_gpu = gpu.step(X, N)
            compare_step(t, O_ref, n_ref, O_gpu, n_gpu)
        assert all(not b.any() for b in gpu.buffers())
    finally:
        gpu.close()
        host.free()


DUALPTR_CASES = [
    # name, batch, K = S, steps, context, retention
    ("k512", 4, 512, 20, 4000, 0.8),
    # the operating points of the matching comparison (Appendix C, Fig. 3a):
    # two and four indices per thread in the freed-slot compaction
    ("k1024_b16", 16, 1024, 48, 65536, 0.9),
    ("k2048_b16", 16, 2048, 48, 65536, 0.9),
]


@pytest.mark.parametrize("name,batch,k,steps,ctx,retention", DUALPTR_CASES, ids=[c[0] for c in DUALPTR_CASES])
def test_dual_pointer_parity(name, batch, k, steps, ctx, retention):
    """Scalar dual-pointer baseline (S = K) against its oracle: slots, miss
    counts and transfer lists every step, buffers every 16 steps."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"dualptr_{name}", batch=batch, topk=k, slots=k, n_q=1, steps=steps,
                         ctx=ctx, retention=retention)
    wl = W.Workload(spec)
    host = HostRows(wl)
    dp = ORC.DualPointerOracle(spec.batch, spec.topk)
    images = [np.zeros((spec.batch, spec.slots, spec.row_bytes[0]), dtype=np.uint8)]
    bptr = [images[0][r].ctypes.data for r in range(spec.batch)]
    gpu = GpuSide(wl, host, match_mode=A.AVSG_MATCH_DUALPTR)
    log(f"[gpu] dual-pointer B={batch} K=S={k} T={steps}")
    try:
        hits = 0
        for t in range(spec.steps):
            X = wl.topk(t)
            O_ref, n_ref = dp.step(X, host=host.ptrs, buf=bptr, row_bytes=list(spec.row_bytes))
            O_gpu, n_gpu = gpu.step(X, None)
            compare_step(t, O_ref, n_ref, O_gpu, n_gpu)
            hits += int(spec.batch * k - n_ref.sum())
            for r in range(spec.batch):
                gx, go = gpu.op.export_misses(r)
                assert np.array_equal(gx, dp.miss_x[r, :n_ref[r, 0]]), f"step {t} request {r} miss ids"
                assert np.array_equal(go, dp.miss_o[r, :n_ref[r, 0]]), f"step {t} request {r} miss slots"
            if t % 16 == 0 or t == spec.steps - 1:
                bufs = gpu.buffers()
                assert np.array_equal(bufs[0], images[0]), f"step {t}: buffers differ"
                content_check(host, wl, bufs, X, O_gpu)
        st = gpu.op.stats()
        assert st["hits"] == hits and st["misses"] == spec.steps * spec.batch * k - hits
    finally:
        gpu.close()
        host.free()


def test_reset_request_and_determinism():
    """A reset request starts cold (token 0 all misses); two runs of the same
    inputs give identical outputs."""
    spec = W.custom_spec(name="reset", batch=3, topk=256, slots=1024, n_q=2, steps=6, ctx=5000)
    outs = []
    for run in range(2):
        wl = W.Workload(spec)
        host = HostRows(wl)
        gpu = GpuSide(wl, host)
        try:
            res = []
            for t in range(spec.steps):
                X = wl.topk(t)
                if t == 4:
                    from paper_2609_37538_amd import avsg as A
                    A.avsg_reset_request(gpu.op.h, 1, gpu.op.stream.cuda_stream)
                O, n = gpu.step(X, wl.verified_len(t))
                res.append((O, n))
                if t == 4:
                    assert n[1, 0] == spec.topk
                    c, q = gpu.op.export_state(1)
                    assert c.max() < spec.ctx
            outs.append(res)
        finally:
            gpu.close()
            host.free()
    for (a, b), (c, d) in zip(outs[0], outs[1]):
        assert np.array_equal(a, c) and np.array_equal(b, d)


def test_bad_indices_are_counted_not_copied():
    """An index outside [0, rows) is counted; its row is not read."""
    from paper_2609_37538_amd import avsg as A
    import torch
    host = A.HostRegion(100 * 16)
    host.view()[:] = 7
    cfg = A.make_config(1, 4, 1, 16, row_bytes=(16,))
    op = A.Operator(cfg, [host.ptr], [100])
    try:
        X = torch.tensor([[[1, 2, 100, 3]]], dtype=torch.int32, device="cuda")
        O, n = op.step(X)
        torch.cuda.synchronize()
        st = op.stats()
        assert st["bad_indices"] == 1 and n.item() == 4
        buf = op.buffers[0].cpu().numpy()[0]
        o = O.cpu().numpy()[0, 0]
        assert np.all(buf[o[[0, 1, 3]]] == 7) and np.all(buf[o[2]] == 0)
    finally:
        op.close()
        host.free()


def test_validate_mode_rejects_bad_selections():
    """Validate mode: a step whose selections hold an index outside [0, rows)
    or an index repeated within one token fails with AVSG_E_BADINDEX before
    any table write (every table unchanged), the error names the first bad
    (request, token) of the oracle's selection check, and the clean steps
    around it equal the oracle's, buffers included."""
    from paper_2609_37538_amd import avsg as A
    import torch
    spec = W.custom_spec(name="validate", batch=4, topk=256, slots=1024, n_q=2, steps=14, ctx=3000,
                         row_bytes=(1152, 132))
    wl = W.Workload(spec)
    host = HostRows(wl)
    orc = OracleSide(wl, host)
    cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, row_bytes=spec.row_bytes,
                        gather_mode=A.AVSG_GATHER_RESIDENT, validate=1)
    op = A.Operator(cfg, host.ptrs, wl.ctx)
    rng = np.random.default_rng(11)
    log("[gpu] validate mode")
    refused = 0
    try:
        for t in range(spec.steps):
            X = wl.topk(t)
            if t % 3 == 1:
                bad = X.copy()
                for _ in range(1 + t % 2):
                    r, g = int(rng.integers(spec.batch)), int(rng.integers(spec.n_q))
                    i, j = rng.choice(spec.topk, size=2, replace=False)
                    kind = (t // 3) % 3
                    if kind == 0:
                        bad[r, g, i] = bad[r, g, j]                  # repeated within the token
                    elif kind == 1:
                        bad[r, g, i] = int(wl.ctx[r])                # one past the last row
                    else:
                        bad[r, g, i] = -3
                verdict = ORC.validate(bad, wl.ctx).ravel()
                first = int(np.flatnonzero(verdict)[0])
                before = [op.export_state(r) for r in range(spec.batch)]
                with pytest.raises(A.AvsgError) as e:
                    op.step(torch.from_numpy(bad).cuda())
                assert e.value.status == A.AVSG_E_BADINDEX
                msg = str(e.value)
                assert f"request {first // spec.n_q} token {first % spec.n_q}:" in msg, msg
                assert ("outside" in msg) == bool(verdict[first] & 1) and \
                       ("repeated" in msg) == bool(verdict[first] & 2), msg
                for r in range(spec.batch):
                    c, q = op.export_state(r)
                    assert np.array_equal(c, before[r][0]) and np.array_equal(q, before[r][1])
                refused += 1
            O_ref, n_ref = orc.step(X, None)
            O_gpu, n_gpu = op.step(torch.from_numpy(X).cuda())
            torch.cuda.synchronize()
            compare_step(t, O_ref, n_ref, O_gpu.cpu().numpy(), n_gpu.cpu().numpy())
        bufs = [b.cpu().numpy() for b in op.buffers]
        for s_ in range(len(spec.row_bytes)):
            assert np.array_equal(bufs[s_], orc.images[s_])
        assert refused == 5 and op.stats()["steps"] == spec.steps
    finally:
        op.close()
        host.free()


def test_import_state_round_trip():
    """A table exported from one handle and imported into another (with the
    buffer bytes copied) continues exactly: both handles and the oracle step
    the same inputs with equal slots, counts, tables and buffers; a lifetime
    outside [-1, L] is refused."""
    from paper_2609_37538_amd import avsg as A
    import torch
    spec = W.custom_spec(name="import", batch=3, topk=256, slots=1024, n_q=2, steps=16, ctx=4000,
                         row_bytes=(1152, 132), retention=0.8)
    wl = W.Workload(spec)
    host = HostRows(wl)
    orc = OracleSide(wl, host)
    gpus = [GpuSide(wl, host, gather_mode=A.AVSG_GATHER_RESIDENT)]
    log("[gpu] export -> import round trip")
    try:
        for t in range(spec.steps):
            X = wl.topk(t)
            if t == 8:
                second = GpuSide(wl, host, gather_mode=A.AVSG_GATHER_RESIDENT)
                for r in range(spec.batch):
                    c, q = gpus[0].op.export_state(r)
                    second.op.import_state(r, c, q)
                for a, b in zip(gpus[0].op.buffers, second.op.buffers):
                    b.copy_(a)
                torch.cuda.synchronize()
                gpus.append(second)
                c, q = gpus[0].op.export_state(0)
                q_bad = q.copy()
                q_bad[5] = (q_bad[5] & 0x00FFFFFF) | (17 << 24)   # lifetime L + 1
                with pytest.raises(A.AvsgError) as e:
                    second.op.import_state(0, c, q_bad)
                assert e.value.status == A.AVSG_E_RANGE
            O_ref, n_ref = orc.step(X, None)
            for gpu in gpus:
                O_gpu, n_gpu = gpu.step(X, None)
                compare_step(t, O_ref, n_ref, O_gpu, n_gpu)
                for r in range(spec.batch):
                    c_ref, q_ref = orc.o.export(r)
                    c_gpu, q_gpu = gpu.op.export_state(r)
                    assert np.array_equal(c_ref, c_gpu) and np.array_equal(q_ref, q_gpu), f"step {t}"
        for gpu in gpus:
            bufs = gpu.buffers()
            for s_ in range(len(spec.row_bytes)):
                assert np.array_equal(bufs[s_], orc.images[s_])
    finally:
        for gpu in gpus:
            gpu.close()
        host.free()


@pytest.mark.parametrize("mix", ["batch64_mtp2", "stress"])
def test_mtp_cold_start_reuse(mix):
    """Cold start with N_q = 1..4 query tokens on the full-batch token mixes
    of batch64_mtp2 and stress (Section 3.6): with one table per request, the
    first token misses every index and the step's slots, counts and hits
    equal the oracle's (later tokens reuse the first token's reservations);
    with an independent table per token nothing hits at step 0."""
    import dataclasses
    import torch
    from paper_2609_37538_amd import avsg as A
    host = A.HostRegion(1 << 16)
    try:
        for n_q in (1, 2, 3, 4):
            spec = dataclasses.replace(W.get_spec(mix), n_q=n_q)
            wl = W.Workload(spec)
            X, N = wl.topk(0), wl.verified_len(0)
            B, K = spec.batch, spec.topk
            log(f"[gpu] cold start {mix} n_q={n_q}")
            for label, b, nq in (("shared", B, n_q), ("independent", B * n_q, 1)):
                Xs = np.ascontiguousarray(X.reshape(b, nq, K))
                ctx = wl.ctx if label == "shared" else np.repeat(wl.ctx, n_q)
                Ns = N if label == "shared" else np.repeat(N, n_q)
                orc = ORC.Oracle(b, K, nq, spec.slots)
                O_ref, n_ref = orc.step(Xs, Ns, rows=ctx)
                cfg = A.make_config(b, K, nq, spec.slots, row_bytes=(16,), gather_mode=A.AVSG_GATHER_NONE)
                op = A.Operator(cfg, [host.ptr] * b, ctx)
                try:
                    O_gpu, n_gpu = op.step(torch.from_numpy(Xs).cuda(), torch.from_numpy(Ns).cuda())
                    torch.cuda.synchronize()
                    compare_step(0, O_ref, n_ref, O_gpu.cpu().numpy(), n_gpu.cpu().numpy())
                    hits = op.stats()["hits"]
                finally:
                    op.close()
                assert hits == orc.total_stats()["hits"]
                assert np.all(n_ref[:, 0] == K)
                if label == "independent" or n_q == 1:
                    assert hits == 0
                else:
                    assert hits > 0.3 * B * (n_q - 1) * K
    finally:
        host.free()


RESIDENT_CASES = [
    # name, kwargs of workload.custom_spec, retry R (R = 0 loses many installs)
    ("lost_installs", dict(batch=4, topk=256, slots=512, n_q=2, steps=24, ctx=3000, retention=0.8), 0),
    ("mtp4_exact_capacity", dict(batch=2, topk=512, slots=2048, n_q=4, steps=16, ctx=20000), 3),
    ("two_streams_odd", dict(batch=3, topk=200, slots=512, n_q=2, steps=12, ctx=9000,
                             row_bytes=(1152, 132)), 1),
    ("spec_window", dict(batch=2, topk=256, slots=2048, n_q=3, steps=20, ctx=4096, mode="zipf_window",
                         window=64, retention=0.8), 3),
    ("k_one", dict(batch=5, topk=1, slots=2, n_q=1, steps=40, ctx=6), 0),
    ("s_16384_max", dict(batch=2, topk=1024, slots=16384, n_q=3, steps=8, ctx=300000), 3),
    ("batch_200", dict(batch=200, topk=128, slots=256, n_q=2, steps=6, ctx=2000), 0),
    ("batch_1024_max", dict(batch=1024, topk=16, slots=64, n_q=2, steps=6, ctx=400), 0),
    ("four_waves", dict(batch=3, topk=384, slots=1024, n_q=2, steps=12, ctx=6000, retention=0.8), 0),
    # the largest plans that fit one workgroup's LDS: with the transfer list
    # and the scan's per-wave candidate lists in LDS (39 tokens), with the
    # transfer list alone (53 tokens; each lane walks its own candidates) and
    # with the list read back from device memory (62 tokens)
    ("lds_edge_scan", dict(batch=2, topk=128, slots=16384, n_q=39, steps=6, ctx=60000), 3),
    ("lds_edge_list", dict(batch=2, topk=128, slots=16384, n_q=53, steps=6, ctx=60000), 3),
    ("lds_edge_no_list", dict(batch=2, topk=128, slots=16384, n_q=62, steps=6, ctx=60000), 3),
]


@pytest.mark.parametrize("name,kw,retry", RESIDENT_CASES, ids=[c[0] for c in RESIDENT_CASES])
def test_resident_reuse_parity(name, kw, retry):
    """Resident-reuse transfer: the plan (host list, device list) equals the
    oracle's transfer_plan bit for bit, and slots, tables, counters and every
    buffer byte equal the oracle's paper-order Stage Two."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"res_{name}", **kw)
    ref, got = run_parity(spec, table_every=4, buffers_every=1, miss_list_requests=3,
                          gather_mode=A.AVSG_GATHER_RESIDENT, retry=retry)
    moved_on_device = (got["resident_rows"] + got["duplicate_rows"]) * sum(spec.row_bytes)
    assert got["host_bytes"] + moved_on_device == got["bytes_moved"]


@pytest.mark.parametrize("workers", [1, 3, 5, 9, 1000])
def test_resident_reuse_worker_counts(workers):
    """Resident-reuse transfer with grids from one workgroup (no workgroup
    starts with the resident list) to more workgroups than rows: every host,
    fan and resident row is still copied exactly once."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"res_workers_{workers}", batch=3, topk=256, slots=512, n_q=2, steps=12,
                         ctx=3000, retention=0.8, row_bytes=(1152, 132))
    ref, got = run_parity(spec, table_every=4, buffers_every=1, miss_list_requests=3,
                          gather_mode=A.AVSG_GATHER_RESIDENT, retry=0, gather_workers=workers)
    assert got["resident_rows"] > 0 and got["duplicate_rows"] > 0


def test_resident_reuse_with_bad_indices():
    """Indices outside [0, rows) stay host entries that the copy skips, and the
    buffers match the balanced transfer's step by step."""
    from paper_2609_37538_amd import avsg as A
    import torch
    rows, S, K = 40, 16, 4
    host = A.HostRegion(rows * 16)
    host.view()[:] = np.repeat(np.arange(rows, dtype=np.uint8), 16)
    ops = [A.Operator(A.make_config(1, K, 2, S, retry=0, max_life=2, row_bytes=(16,), gather_mode=gm),
                      [host.ptr], [rows])
           for gm in (A.AVSG_GATHER_BALANCED, A.AVSG_GATHER_RESIDENT)]
    rng = np.random.default_rng(5)
    try:
        for t in range(12):
            X = np.stack([rng.choice(rows + 8, size=K, replace=False) for _ in range(2)])
            X[1, :2] = X[0, :2]                  # repeats across the two tokens
            Xd = torch.tensor(X[None], dtype=torch.int32, device="cuda")
            outs = [op.step(Xd) for op in ops]
            torch.cuda.synchronize()
            assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])
            assert torch.equal(ops[0].buffers[0], ops[1].buffers[0]), f"step {t}"
            hx, ho, hf, rs, rd, ps, pd = ops[1].export_plan(0)
            mx, _ = ops[1].export_misses(0)
            assert sorted(hx[hx >= rows].tolist()) == sorted(mx[mx >= rows].tolist())
        st = ops[1].stats()
        assert st["bad_indices"] > 0 and st["resident_rows"] + st["duplicate_rows"] > 0
    finally:
        for op in ops:
            op.close()
        host.free()


def test_resident_reuse_refused_without_room():
    """The plan's index map must fit beside the table in LDS, and the mode
    needs hash matching."""
    from paper_2609_37538_amd import avsg as A
    chk = lambda **kw: A.avsg_check_config(A.make_config(**kw))
    assert chk(batch=1, topk=128, n_q=62, slots=16384, row_bytes=(16,),
               gather_mode=A.AVSG_GATHER_RESIDENT) == A.AVSG_OK
    assert chk(batch=1, topk=128, n_q=63, slots=16384, row_bytes=(16,),
               gather_mode=A.AVSG_GATHER_RESIDENT) == A.AVSG_E_CAPACITY
    assert chk(batch=1, topk=128, n_q=110, slots=16384, row_bytes=(16,)) == A.AVSG_OK
    assert chk(batch=1, topk=64, n_q=1, slots=64, row_bytes=(16,), match_mode=A.AVSG_MATCH_DUALPTR,
               gather_mode=A.AVSG_GATHER_RESIDENT) == A.AVSG_E_UNSUPPORTED


PIPELINED_CASES = [
    ("tiny", None),
    ("mtp3_ragged", dict(batch=5, topk=300, slots=1024, n_q=3, steps=12, ctx=8000, row_bytes=(1152, 132))),
    ("all_hits", dict(batch=2, topk=256, slots=1024, n_q=2, steps=8, ctx=256, retention=1.0, overlap=1.0)),
    ("spec_window", dict(batch=3, topk=256, slots=2048, n_q=3, steps=16, ctx=4096, mode="zipf_window",
                         window=64, retention=0.8)),
]


@pytest.mark.parametrize("name,kw", PIPELINED_CASES, ids=[c[0] for c in PIPELINED_CASES])
def test_pipelined_step_parity(name, kw):
    """Stage One and Stage Two in one launch (chunk queue): same outputs,
    tables, counters and buffers as the oracle, and no queue time-outs."""
    spec = W.get_spec("tiny") if kw is None else W.custom_spec(name=name, **kw)
    ref, got = run_parity(spec, table_every=2, buffers_every=2, miss_list_requests=2, gather_mode=5)
    assert got["queue_timeouts"] == 0


def test_pipelined_batch_limit():
    """The pipelined step needs every request's producer resident: batch above
    the CU count is refused at create time."""
    from paper_2609_37538_amd import avsg as A
    cus = A.avsg_device_cus()
    B = cus + 1
    host = A.HostRegion(B * 64 * 16)
    cfg = A.make_config(B, 16, 1, 64, row_bytes=(16,), gather_mode=A.AVSG_GATHER_PIPELINED)
    try:
        with pytest.raises(A.AvsgError) as e:
            A.Operator(cfg, [host.ptr + r * 64 * 16 for r in range(B)], [64] * B)
        assert e.value.status == A.AVSG_E_UNSUPPORTED
    finally:
        host.free()


# ---- the five benchmark workloads at full size ----------------------------
@pytest.mark.timeout(900)
def test_parity_batch16_full():
    """Batch 16 at full size with the paper's Stage Two (S3), resident reuse and
    the early fetch stepped side by side on the same inputs."""
    ref, got = run_parity_modes(W.get_spec("batch16"), (0, 6, 7))
    assert got[6]["resident_rows"] > 0 and got[7]["early_rows"] > 0


@pytest.mark.timeout(900)
def test_parity_batch64_mtp2_full():
    run_parity(W.get_spec("batch64_mtp2"))


@pytest.mark.timeout(900)
def test_parity_batch64_mtp2_full_pipelined():
    ref, got = run_parity(W.get_spec("batch64_mtp2"), gather_mode=5)
    assert got["queue_timeouts"] == 0


@pytest.mark.timeout(900)
def test_parity_batch64_mtp2_full_resident():
    from paper_2609_37538_amd import avsg as A
    ref, got = run_parity(W.get_spec("batch64_mtp2"), gather_mode=A.AVSG_GATHER_RESIDENT)
    assert got["host_bytes"] < 0.8 * got["bytes_moved"]


@pytest.mark.timeout(900)
def test_parity_batch64_mtp2_full_early():
    from paper_2609_37538_amd import avsg as A
    ref, got = run_parity(W.get_spec("batch64_mtp2"), gather_mode=A.AVSG_GATHER_EARLY)
    assert got["early_rows"] > 0.95 * (got["host_bytes"] // sum(W.get_spec("batch64_mtp2").row_bytes))


@pytest.mark.timeout(900)
def test_parity_imbalance_full():
    """The load-imbalance workload at full size (32 requests whose miss counts
    differ by more than 10x): CU-balanced (S3, Eq. 6) against request-level
    (S1, Eq. 13) and position-level (S2, Eq. 14) transfer, plus resident reuse
    and the early fetch, all stepped on the same inputs and each compared with
    the oracle element by element."""
    ref, got = run_parity_modes(W.get_spec("imbalance"), (0, 1, 4, 6, 7))
    assert got[6]["resident_rows"] > 0 and got[7]["early_rows"] > 0


@pytest.mark.timeout(1200)
def test_parity_stress_full():
    ref, got = run_parity(W.get_spec("stress"), buffers_every=128)
    assert got["invalidations"] > 0


@pytest.mark.timeout(1200)
def test_parity_stress_full_early():
    """Speculative rows are rewritten every step: an index cached at or above
    the verified length is never an early key (some slot holds it), and an
    early row is read from the host during the step it is listed in."""
    from paper_2609_37538_amd import avsg as A
    ref, got = run_parity(W.get_spec("stress"), buffers_every=64, gather_mode=A.AVSG_GATHER_EARLY)
    assert got["invalidations"] > 0 and got["early_rows"] > 0


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("mode", [0, 6], ids=["balanced", "resident"])
def test_parity_stress_four_tokens(mode):
    """The stress mix with four query tokens per step (three draft tokens):
    the four tokens' reservations fill the whole table (N_q K = S, Eq. 7), so
    every slot the step did not refresh may be reclaimed; 192 steps at full
    size (32 requests, K = 2048, S = 8192, 1M-token contexts)."""
    ref, got = run_parity(W.get_spec("stress_mtp3"), steps=192, buffers_every=64, gather_mode=mode)
    assert got["invalidations"] > 0
    if mode == 6:
        assert got["resident_rows"] > 0


@pytest.mark.timeout(1200)
def test_parity_stress_full_resident():
    """Speculative rows are rewritten every step: the plan must never reuse a
    slot whose cached index was invalidated."""
    from paper_2609_37538_amd import avsg as A
    ref, got = run_parity(W.get_spec("stress"), buffers_every=64, gather_mode=A.AVSG_GATHER_RESIDENT)
    assert got["invalidations"] > 0 and got["resident_rows"] > 0


EARLY_CASES = [
    # name, kwargs of workload.custom_spec, retry R, staging rows, direct writes (0 on, -1 off)
    ("lost_installs", dict(batch=4, topk=256, slots=512, n_q=2, steps=24, ctx=3000, retention=0.8), 0, 0, 0),
    ("mtp4_exact_capacity", dict(batch=2, topk=512, slots=2048, n_q=4, steps=16, ctx=20000), 3, 0, 0),
    ("mtp5_capped_keys", dict(batch=2, topk=64, slots=512, n_q=5, steps=16, ctx=400, overlap=0.9), 0, 0, 0),
    ("two_streams_odd", dict(batch=3, topk=200, slots=512, n_q=2, steps=12, ctx=9000,
                             row_bytes=(1152, 132)), 1, 0, 0),
    ("spec_window", dict(batch=2, topk=256, slots=2048, n_q=3, steps=20, ctx=4096, mode="zipf_window",
                         window=64, retention=0.8), 3, 0, 0),
    ("k_one", dict(batch=5, topk=1, slots=2, n_q=1, steps=40, ctx=6), 0, 0, 0),
    ("s_16384_max", dict(batch=2, topk=1024, slots=16384, n_q=3, steps=8, ctx=300000), 3, 0, 0),
    ("batch_200", dict(batch=200, topk=128, slots=256, n_q=2, steps=6, ctx=2000), 0, 0, 0),
    ("batch_1024_max", dict(batch=1024, topk=16, slots=64, n_q=2, steps=6, ctx=400), 0, 0, 0),
    ("four_waves", dict(batch=3, topk=384, slots=1024, n_q=2, steps=12, ctx=6000, retention=0.8), 0, 0, 0),
    ("all_staged", dict(batch=4, topk=256, slots=512, n_q=2, steps=12, ctx=3000, retention=0.8,
                        row_bytes=(1152, 132)), 0, 0, -1),
    ("all_deferred", dict(batch=4, topk=256, slots=512, n_q=2, steps=12, ctx=3000, retention=0.8,
                          row_bytes=(1152, 132)), 0, -1, -1),
    ("five_staging_rows", dict(batch=4, topk=256, slots=1024, n_q=3, steps=12, ctx=3000, retention=0.8,
                               row_bytes=(1152, 132)), 0, 5, -1),
]


@pytest.mark.parametrize("name,kw,retry,staging,direct", EARLY_CASES, ids=[c[0] for c in EARLY_CASES])
def test_early_fetch_parity(name, kw, retry, staging, direct):
    """Early-fetch transfer: the early list equals the oracle's early_set (keys
    and positions), the plan of the remaining misses equals
    transfer_plan_early, and slots, tables, counters and every buffer byte
    equal the oracle's paper-order Stage Two, with rows written straight into
    their slots, parked in staging, or re-read from the host after Stage One."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"early_{name}", **kw)
    ref, got = run_parity(spec, table_every=4, buffers_every=1, miss_list_requests=3,
                          gather_mode=A.AVSG_GATHER_EARLY, retry=retry, early_staging_rows=staging,
                          early_direct=direct)
    moved_on_device = (got["resident_rows"] + got["duplicate_rows"]) * sum(spec.row_bytes)
    assert got["host_bytes"] + moved_on_device == got["bytes_moved"]
    assert got["early_rows"] > 0
    if direct == -1:
        assert got["early_staged_rows"] + got["early_deferred_rows"] == got["early_rows"]
        if staging == -1:
            assert got["early_deferred_rows"] == got["early_rows"]
        if staging == 5:
            assert got["early_staged_rows"] > 0 and got["early_deferred_rows"] > 0


@pytest.mark.parametrize("workers", [1, 3, 1000])
def test_early_fetch_worker_counts(workers):
    """Early-fetch transfer with one, a few and more copy workgroups than
    early rows: every early row is copied exactly once into every slot of its
    positions."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name=f"early_workers_{workers}", batch=3, topk=256, slots=512, n_q=2, steps=12,
                         ctx=3000, retention=0.8, row_bytes=(1152, 132))
    ref, got = run_parity(spec, table_every=4, buffers_every=1, miss_list_requests=3,
                          gather_mode=A.AVSG_GATHER_EARLY, retry=0, gather_workers=workers)
    assert got["early_rows"] > 0 and got["duplicate_rows"] > 0


@pytest.mark.parametrize("mode", [0, 6], ids=["balanced", "resident"])
def test_layer_batching_matches_per_layer_steps(mode):
    """Multi-layer batching: every (layer, request) pair owns its table,
    buffer and host rows, so one launch over three layers of two requests
    gives the slots, counts and buffer bytes of one step per layer, and both
    equal the oracle."""
    from paper_2609_37538_amd import avsg as A
    import torch
    layers, per = 3, 2
    spec = W.custom_spec(name=f"layers_{mode}", batch=layers * per, topk=256, slots=1024, n_q=2, steps=10,
                         ctx=5000, retention=0.8, row_bytes=(1152, 132))
    wl = W.Workload(spec)
    host = HostRows(wl)
    orc = OracleSide(wl, host, retry=1)
    B, ns = spec.batch, len(spec.row_bytes)
    kw = dict(retry=1, row_bytes=spec.row_bytes, gather_mode=mode)
    one = A.Operator(A.make_config(B, spec.topk, spec.n_q, spec.slots, **kw), host.ptrs, wl.ctx)
    each = [A.Operator(A.make_config(per, spec.topk, spec.n_q, spec.slots, **kw),
                       [host.ptrs[s * B + l * per + i] for s in range(ns) for i in range(per)],
                       wl.ctx[l * per:(l + 1) * per]) for l in range(layers)]
    try:
        for t in range(spec.steps):
            X = wl.topk(t)
            O_ref, n_ref = orc.step(X, None)
            Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.int32)).cuda()
            one.step(Xd)
            for l, op in enumerate(each):
                op.step(Xd[l * per:(l + 1) * per])
            torch.cuda.synchronize()
            compare_step(t, O_ref, n_ref, one.slots.cpu().numpy(), one.miss_counts.cpu().numpy())
            for l, op in enumerate(each):
                sl = slice(l * per, (l + 1) * per)
                assert torch.equal(one.slots[sl], op.slots) and torch.equal(one.miss_counts[sl], op.miss_counts)
                for s in range(ns):
                    assert torch.equal(one.buffers[s][sl], op.buffers[s]), f"step {t} layer {l} stream {s}"
            for s in range(ns):
                assert np.array_equal(one.buffers[s].cpu().numpy(), orc.images[s]), f"step {t} stream {s}"
    finally:
        one.close()
        for op in each:
            op.close()
        host.free()


@pytest.mark.parametrize("early", [False, True], ids=["resident", "early"])
def test_resident_reuse_when_verified_length_shrinks(early):
    """A verified length that moves back: slots caching an index at or above
    the current verified length are never plan sources (the oracle sees them
    invalidated), while the speculative rows beyond the largest length so far
    are rewritten every step; plans, slots and buffers equal the oracle's, and
    the case is exercised (such an index misses while a slot still caches it).
    With the early fetch, indices no slot caches at the start of a step
    (speculative ones among them) are read from the rows as rewritten for that
    step, and the early sets equal the oracle's."""
    from paper_2609_37538_amd import avsg as A
    spec = W.custom_spec(name="shrink_n", batch=2, topk=64, slots=512, n_q=2, steps=16, ctx=4096)
    wl = W.Workload(spec)
    host = HostRows(wl)
    orc = OracleSide(wl, host, retry=0, max_life=8)
    mode = A.AVSG_GATHER_EARLY if early else A.AVSG_GATHER_RESIDENT
    gpu = GpuSide(wl, host, retry=0, max_life=8, gather_mode=mode)
    early_spec = 0
    rng = np.random.default_rng(11)
    n_max = 0
    exercised = 0
    try:
        for t in range(spec.steps):
            n_t = 2000 + 4 * t if t < 8 else 2000 + 32 - 8 * (t - 7)   # grows, then moves back
            n_max = max(n_max, n_t)
            N = np.full(spec.batch, n_t, dtype=np.int64)
            for s in range(len(spec.row_bytes)):
                for r in range(spec.batch):
                    rows = host.row_view(s, r)[n_max:n_max + 16]    # never verified so far
                    rows[:] = rng.integers(0, 256, size=rows.shape, dtype=np.uint8)
            X = np.empty((spec.batch, spec.n_q, spec.topk), dtype=np.int32)
            for r in range(spec.batch):
                others = rng.choice(n_t - 24, size=spec.topk - 40, replace=False)
                for g in range(spec.n_q):
                    X[r, g] = np.concatenate([np.arange(n_t - 24, n_t + 16), others])
            cached = [orc.o.export(r)[0] for r in range(spec.batch)]
            O_ref, n_ref = orc.step(X, N)
            O_gpu, n_gpu = gpu.step(X, N)
            compare_step(t, O_ref, n_ref, O_gpu, n_gpu)
            bufs = gpu.buffers()
            for s in range(len(spec.row_bytes)):
                assert np.array_equal(bufs[s], orc.images[s]), f"step {t} stream {s}: buffers differ"
            content_check(host, wl, bufs, X, O_gpu)
            for r in range(spec.batch):
                mx, mo = orc.o.misses(r, n_ref[r])
                c_ref, _ = orc.o.export(r)
                if early:
                    keys, where = ORC.early_set(X[r], cached[r], int(wl.ctx[r]))
                    gk, gpos = gpu.op.export_early(r)
                    order = np.argsort(gk, kind="stable")
                    assert np.array_equal(gk[order], keys), f"step {t} request {r}: early keys differ"
                    for k, ps in enumerate(where):
                        got_ps = sorted(int(v) for v in gpos[order[k]] if v >= 0)
                        assert got_ps == ps, f"step {t} request {r}: positions of {keys[k]} differ"
                    early_spec += int(np.sum(keys >= n_t))
                    want = ORC.transfer_plan_early(mx, mo, c_ref, int(wl.ctx[r]), keys)
                else:
                    want = ORC.transfer_plan(mx, mo, c_ref, int(wl.ctx[r]))
                got = gpu.op.export_plan(r)
                for k in range(7):
                    assert np.array_equal(want[k], got[k]), f"step {t} request {r}: plan list {k}"
                reserved = set(mo.tolist())
                for x in mx.tolist():
                    if x >= n_t and any(cached[r][j] == x and j not in reserved for j in range(spec.slots)):
                        exercised += 1
        st = gpu.op.stats()
        assert exercised > 0 and st["invalidations"] > 0
        assert st["resident_rows"] + st["duplicate_rows"] > 0
        if early:
            assert early_spec > 0 and st["early_rows"] > 0
    finally:
        gpu.close()
        host.free()


def test_two_handles_on_two_streams():
    """Three handles (balanced, resident-reuse and early-fetch Stage Two, each
    with its own workspace and buffers) step the same selections on two
    streams with no synchronization between them; slots, counts, tables and
    buffers of all three equal the oracle's after every step."""
    from paper_2609_37538_amd import avsg as A
    import torch
    spec = W.custom_spec(name="two_streams", batch=6, topk=512, slots=2048, n_q=2, steps=10,
                         ctx=30000, row_bytes=(1152, 132), retention=0.8)
    wl = W.Workload(spec)
    host = HostRows(wl)
    orc = OracleSide(wl, host, retry=1)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    streams.append(streams[0])
    ops = []
    try:
        for gm, st in zip((A.AVSG_GATHER_BALANCED, A.AVSG_GATHER_RESIDENT, A.AVSG_GATHER_EARLY), streams):
            cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, retry=1,
                                row_bytes=spec.row_bytes, gather_mode=gm)
            ops.append(A.Operator(cfg, host.ptrs, wl.ctx, stream=st))
        for t in range(spec.steps):
            X = wl.topk(t)
            log(f"[two streams] step {t}")
            Xd = torch.from_numpy(np.ascontiguousarray(X, dtype=np.int32)).cuda()
            torch.cuda.synchronize()
            for op, st in zip(ops, streams):
                with torch.cuda.stream(st):
                    op.step(Xd)
            O_ref, n_ref = orc.step(X, None)
            torch.cuda.synchronize()
            for op in ops:
                compare_step(t, O_ref, n_ref, op.slots.cpu().numpy(), op.miss_counts.cpu().numpy())
                bufs = [b.cpu().numpy() for b in op.buffers]
                for s in range(len(spec.row_bytes)):
                    assert np.array_equal(bufs[s], orc.images[s]), f"step {t} stream {s}: buffers differ"
        for r in range(spec.batch):
            c_ref, q_ref = orc.o.export(r)
            for op in ops:
                c_gpu, q_gpu = op.export_state(r)
                assert np.array_equal(c_ref, c_gpu) and np.array_equal(q_ref, q_gpu)
    finally:
        for op in ops:
            op.close()
        host.free()


@pytest.mark.parametrize("mode,n_q", [(0, 2), (1, 1), (4, 2), (5, 2), (6, 2), (6, 3), (7, 2), (7, 3)],
                         ids=["balanced", "request_level", "position_level", "pipelined", "resident",
                              "resident_3_tokens", "early", "early_3_tokens"])
def test_graph_capture_replays_steps(mode, n_q):
    """One avsg_step captured into a HIP graph and replayed once per decode
    step (new selections copied into the captured input between replays, with
    host synchronizations): after every replay the slots, counts and buffers
    equal an operator stepped eagerly on the same selections, and at the end
    so do the tables and counters."""
    from paper_2609_37538_amd import avsg as A
    import torch
    spec = W.custom_spec(name=f"graph_{mode}_{n_q}", batch=4, topk=256, slots=1024, n_q=n_q, steps=12,
                         ctx=6000, row_bytes=(1152, 132), retention=0.8)
    wl = W.Workload(spec)
    host = HostRows(wl)
    cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, retry=0, max_life=8,
                        row_bytes=spec.row_bytes, gather_mode=mode)
    eager = A.Operator(cfg, host.ptrs, wl.ctx, stream=torch.cuda.Stream())
    graphed = A.Operator(cfg, host.ptrs, wl.ctx, stream=torch.cuda.Stream())
    X_in = torch.zeros((spec.batch, spec.n_q, spec.topk), dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    try:
        with torch.cuda.graph(g, stream=graphed.stream):
            graphed.step(X_in)
        torch.cuda.synchronize()
        assert graphed.stats()["steps"] == 1 and graphed.stats()["lookups"] > 0
        for t in range(spec.steps):
            log(f"[graph] mode {mode} n_q {n_q} replay {t}")
            X = torch.from_numpy(np.ascontiguousarray(wl.topk(t), dtype=np.int32)).cuda()
            X_in.copy_(X)
            torch.cuda.synchronize()
            g.replay()
            eager.step(X)
            torch.cuda.synchronize()
            assert torch.equal(graphed.slots, eager.slots), f"replay {t}: slots differ"
            assert torch.equal(graphed.miss_counts, eager.miss_counts), f"replay {t}: counts differ"
            for b1, b2 in zip(graphed.buffers, eager.buffers):
                assert torch.equal(b1, b2), f"replay {t}: buffers differ"
        for r in range(spec.batch):
            c1, q1 = graphed.export_state(r)
            c2, q2 = eager.export_state(r)
            assert np.array_equal(c1, c2) and np.array_equal(q1, q2)
        s1, s2 = graphed.stats(), eager.stats()
        for k in ("hits", "misses", "lost_exhausted", "lost_collision", "resident_rows", "duplicate_rows",
                  "early_rows"):
            assert s1[k] == s2[k], k
        assert s2["misses"] > 0
    finally:
        del g
        eager.close()
        graphed.close()
        host.free()


@pytest.mark.parametrize("mode", [0, 5, 6, 7], ids=["balanced", "pipelined", "resident", "early"])
def test_graph_of_several_steps(mode):
    """Eight consecutive steps (each one's selections and verified lengths
    copied into the captured inputs, then avsg_step) captured as one HIP graph
    and replayed once after an eager warmup: slots, counts, buffers, tables and
    counters equal an operator stepped eagerly through the same steps."""
    from paper_2609_37538_amd import avsg as A
    import torch
    spec = W.custom_spec(name=f"graph_seq_{mode}", batch=3, topk=256, slots=1024, n_q=2, steps=12,
                         ctx=6000, row_bytes=(1152, 132), retention=0.8)
    wl = W.Workload(spec)
    host = HostRows(wl)
    cfg = A.make_config(spec.batch, spec.topk, spec.n_q, spec.slots, retry=1, max_life=8,
                        row_bytes=spec.row_bytes, gather_mode=mode)
    eager = A.Operator(cfg, host.ptrs, wl.ctx, stream=torch.cuda.Stream())
    graphed = A.Operator(cfg, host.ptrs, wl.ctx, stream=torch.cuda.Stream())
    Xs = torch.from_numpy(np.ascontiguousarray(wl.all_steps(spec.steps), dtype=np.int32)).cuda()
    Ns = torch.from_numpy(np.stack([np.asarray(wl.ctx, dtype=np.int64) - (spec.steps - t)
                                    for t in range(spec.steps)])).cuda()
    X_in, N_in = torch.empty_like(Xs[0]), torch.empty_like(Ns[0])
    g = torch.cuda.CUDAGraph()
    try:
        for t in range(4):
            eager.step(Xs[t], Ns[t])
            graphed.step(Xs[t], Ns[t])
        torch.cuda.synchronize()
        with torch.cuda.graph(g, stream=graphed.stream):
            for t in range(4, spec.steps):
                X_in.copy_(Xs[t])
                N_in.copy_(Ns[t])
                graphed.step(X_in, N_in)
        torch.cuda.synchronize()
        log(f"[graph] mode {mode}: eight captured steps")
        g.replay()
        for t in range(4, spec.steps):
            eager.step(Xs[t], Ns[t])
        torch.cuda.synchronize()
        assert torch.equal(graphed.slots, eager.slots) and torch.equal(graphed.miss_counts, eager.miss_counts)
        for b1, b2 in zip(graphed.buffers, eager.buffers):
            assert torch.equal(b1, b2)
        for r in range(spec.batch):
            c1, q1 = graphed.export_state(r)
            c2, q2 = eager.export_state(r)
            assert np.array_equal(c1, c2) and np.array_equal(q1, q2)
        s1, s2 = graphed.stats(), eager.stats()
        for k in ("hits", "misses", "lost_exhausted", "lost_collision", "invalidations", "resident_rows",
                  "duplicate_rows", "early_rows", "host_bytes"):
            assert s1[k] == s2[k], k
        assert s2["misses"] > 0 and s2["invalidations"] > 0
    finally:
        del g
        eager.close()
        graphed.close()
        host.free()


def test_copy_engine_batched_call_without_torch():
    """In a process that never loads torch, the copy-engine transfer issues one
    batched runtime copy call per step and matches the oracle step by step
    (tests/copy_engine_batched_check.py, run as a child process)."""
    import subprocess
    import sys
    here = os.path.dirname(os.path.abspath(__file__))
    r = subprocess.run([sys.executable, "-u", os.path.join(here, "copy_engine_batched_check.py")],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert r.stdout.strip().splitlines()[-1].startswith("ok copy_calls=")


@pytest.fixture(scope="module")
def c_abi_program(tmp_path_factory):
    """tests/c_abi_parity.c built with gcc against include/avsg.h, the
    library, the C oracle and the HIP runtime."""
    import shutil
    import subprocess
    cc = shutil.which("gcc")
    if cc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = str(tmp_path_factory.mktemp("c_abi") / "c_abi_parity")
    pkg, orc = os.path.join(root, "paper_2609_37538_amd"), os.path.join(root, "oracle")
    subprocess.run([cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
                    "-I", "/opt/rocm/include", "-I", os.path.join(root, "include"), "-I", orc,
                    os.path.join(root, "tests", "c_abi_parity.c"), "-o", exe,
                    "-L", pkg, "-lavsg", "-L", orc, "-loracle_avsg", "-L", "/opt/rocm/lib", "-lamdhip64",
                    f"-Wl,-rpath,{pkg}", f"-Wl,-rpath,{orc}", "-Wl,-rpath,/opt/rocm/lib"], check=True)
    return exe


@pytest.mark.parametrize("mode", [0, 1, 2, 4, 5, 6, 7],
                         ids=["balanced", "request_level", "copy_engine", "position_level", "pipelined",
                              "resident", "early"])
def test_c_caller_against_c_oracle(c_abi_program, mode):
    """A C program drives the library through include/avsg.h (hipMalloc'd
    device memory, its own stream) and the oracle through its C interface;
    slots, counts and both streams' buffers agree after every step."""
    import subprocess
    log(f"[c abi] mode {mode}")
    r = subprocess.run([c_abi_program, str(mode)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-2000:])
    assert r.stdout.startswith(f"ok mode {mode} ")
