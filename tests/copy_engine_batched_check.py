"""Copy-engine transfer with the HIP runtime's batched copy call.

Run as its own process, which must never import torch: the system HIP runtime
then serves the process and exports the batched copy call that the runtime
PyTorch ships lacks.  A small two-stream workload steps through the library
(device memory from hipMalloc) and through the CPU oracle; after every step
the slots, miss counts and every buffer byte must be equal, and the transfer
must have used one runtime copy call per step.  Prints "ok" and the call
count on success; any mismatch raises.
"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

import numpy as np  # noqa: E402

from paper_2609_37538_amd import avsg as A  # noqa: E402

A.load(share_torch_runtime=False)

import bench  # noqa: E402
import workload as W  # noqa: E402
from harness import HostRows, OracleSide  # noqa: E402


def main():
    assert "torch" not in sys.modules
    spec = W.custom_spec(name="copy_engine_batched", batch=3, topk=256, slots=1024, n_q=2, steps=8,
                         ctx=6000, row_bytes=(1152, 132), retention=0.8)
    wl = W.Workload(spec)
    B, K, nq, S = spec.batch, spec.topk, spec.n_q, spec.slots
    host = HostRows(wl)
    orc = OracleSide(wl, host, retry=3)
    hip = bench._Hip()
    cfg = A.make_config(B, K, nq, S, retry=3, row_bytes=spec.row_bytes, gather_mode=A.AVSG_GATHER_SDMA)
    ws_bytes = A.avsg_workspace_bytes(cfg)
    ws = hip.alloc(ws_bytes)
    bases = [hip.alloc(B * S * rb) for rb in spec.row_bytes]
    bufs = [bases[s] + r * S * rb for s, rb in enumerate(spec.row_bytes) for r in range(B)]
    Xd = hip.alloc(B * nq * K * 4)
    slots = hip.alloc(B * nq * K * 4)
    counts = hip.alloc(B * nq * 4)
    stream = hip.stream()           # the batched call refuses the legacy default stream
    h = A.avsg_create(cfg, host.ptrs, wl.ctx, ws, ws_bytes, bufs, stream)
    try:
        for t in range(spec.steps):
            X = np.ascontiguousarray(wl.topk(t), dtype=np.int32)
            hip.upload(Xd, X)
            A.avsg_step(h, Xd, None, slots, counts, stream)
            O_ref, n_ref = orc.step(X, None)
            hip.sync()
            O = np.empty((B, nq, K), dtype=np.int32)
            n = np.empty((B, nq), dtype=np.int32)
            hip.download(O, slots)
            hip.download(n, counts)
            assert np.array_equal(O, O_ref), f"step {t}: slots differ"
            assert np.array_equal(n, n_ref), f"step {t}: miss counts differ"
            for s, rb in enumerate(spec.row_bytes):
                got = np.empty((B, S, rb), dtype=np.uint8)
                hip.download(got, bases[s])
                assert np.array_equal(got, orc.images[s]), f"step {t} stream {s}: buffers differ"
        st = A.avsg_stats(h)
    finally:
        A.avsg_destroy(h)
        hip.free_all()
        host.free()
    assert st["misses"] > 0
    assert st["copy_calls"] == spec.steps, f"expected one batched call per step, got {st['copy_calls']}"
    print(f"ok copy_calls={st['copy_calls']} misses={st['misses']}", flush=True)


if __name__ == "__main__":
    main()
