"""Seeded synthetic decode-step workloads for the AVSG sparse-gather operator.

This package produces inputs only: per-step top-K index matrices, verified
context lengths and host-resident KV / indexer-key rows.  It contains none of
the operator's arithmetic (no hashing, matching, slot choice or transfer
logic), so the CPU oracle and the GPU path can both consume what it produces
without sharing any of the method's code.

The paper's workloads (real per-layer DSA traces of production requests) are
not available; these generators stand in for them with the shapes the paper
uses (top-K = 2048, 4K/8K-slot buffers, 1,152-byte MLA rows of
(512 + 64) bf16 values, MTP up to 3) and an explicit step-to-step retention
process.  Randomness comes from NumPy's counter-based Philox generator keyed by
(seed, config id, request, step, token, purpose), so any step of any request
can be regenerated independently of the others.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libavsg_workload.so")

KV_ROW_BYTES = 1152        # (512 + 64) bf16 values of one MLA latent KV row
INDEXER_ROW_BYTES = 132    # 128 fp8 indexer-key bytes + one fp32 scale


@dataclasses.dataclass(frozen=True)
class Spec:
    """Shape and statistics of one synthetic workload."""

    name: str
    cfg_id: int
    batch: int
    topk: int
    slots: int
    n_q: int
    steps: int
    seed: int = 0
    ctx: int = 8192                       # context (host rows) per request
    ctx_log_uniform: Optional[tuple] = None  # (lo, hi): per-request log-uniform ctx
    retention: float = 0.9                # step-to-step keep probability
    retention_range: Optional[tuple] = None  # (lo, hi): per-request U[lo, hi]
    overlap: float = 0.95                 # tokens g >= 1 share this fraction with token 0
    mode: str = "uniform"                 # "uniform" | "zipf_window" | "controlled"
    zipf_s: float = 1.1
    window: int = 512
    row_bytes: tuple = (KV_ROW_BYTES,)

    @property
    def speculative(self) -> bool:
        return self.mode == "zipf_window" and self.n_q > 1


# The five benchmark workloads.  Sizes, retention and mixes follow the
# operator's decode-step setting: K = 2048 selected tokens per query token,
# 8K-slot buffers, 1,152-byte rows, MTP tokens sharing one buffer.
SPECS = {
    "tiny": Spec("tiny", 0, batch=1, topk=256, slots=1024, n_q=1, steps=64,
                 ctx=8192, retention=0.9),
    "batch16": Spec("batch16", 1, batch=16, topk=2048, slots=8192, n_q=1, steps=256,
                    ctx=65536, retention=0.9),
    "batch64_mtp2": Spec("batch64_mtp2", 2, batch=64, topk=2048, slots=8192, n_q=2,
                         steps=256, ctx=131072, retention=0.9, overlap=0.95,
                         row_bytes=(KV_ROW_BYTES, INDEXER_ROW_BYTES)),
    "imbalance": Spec("imbalance", 3, batch=32, topk=2048, slots=8192, n_q=1, steps=128,
                      ctx_log_uniform=(4096, 1 << 20), retention_range=(0.5, 0.99)),
    "stress": Spec("stress", 4, batch=32, topk=2048, slots=8192, n_q=3, steps=512,
                   ctx=1 << 20, retention=0.8, mode="zipf_window", zipf_s=1.1, window=512),
    # the stress mix with three draft tokens (four query tokens per step): the
    # table holds exactly N_q * K = S reservations, the tightest case of Eq. 7
    "stress_mtp3": Spec("stress_mtp3", 5, batch=32, topk=2048, slots=8192, n_q=4, steps=512,
                        ctx=1 << 20, retention=0.8, mode="zipf_window", zipf_s=1.1, window=512),
}


def get_spec(name: str) -> Spec:
    return SPECS[name]


def custom_spec(name: str = "custom", cfg_id: int = 100, **kw) -> Spec:
    """A spec for tests: any Spec field may be overridden."""
    base = dict(batch=2, topk=64, slots=256, n_q=1, steps=8, ctx=1024)
    base.update(kw)
    return Spec(name, cfg_id, **base)


def _rng(spec: Spec, *key: int) -> np.random.Generator:
    ss = np.random.SeedSequence([spec.seed, spec.cfg_id, *[int(k) for k in key]])
    return np.random.Generator(np.random.Philox(ss))


# purposes, used as the last component of a generator key
_P_CTX, _P_RET, _P_INIT, _P_KEEP, _P_REDRAW, _P_TOKEN, _P_PERM, _P_ZMAP = range(8)


def _draw_excluding(rng: np.random.Generator, lo: int, hi: int, need: int,
                    exclude: np.ndarray) -> np.ndarray:
    """`need` distinct integers uniform on [lo, hi) minus `exclude` (rejection)."""
    out = np.empty(0, dtype=np.int64)
    if need <= 0:
        return out
    excl = np.asarray(exclude, dtype=np.int64)
    avail = (hi - lo) - np.count_nonzero((excl >= lo) & (excl < hi))
    if need > avail:
        raise ValueError(f"cannot draw {need} distinct values from {avail}")
    while out.size < need:
        cand = rng.integers(lo, hi, size=max(2 * (need - out.size), 64), dtype=np.int64)
        _, first = np.unique(cand, return_index=True)
        cand = cand[np.sort(first)]
        cand = cand[~np.isin(cand, excl)]
        cand = cand[~np.isin(cand, out)]
        out = np.concatenate([out, cand[: need - out.size]])
    return out


class Workload:
    """Step-by-step generator of top-K index matrices X[B][n_q][K] (int32).

    Steps must be requested in order 0, 1, 2, ...; step t of request r depends
    on step t-1 of the same request only through the retained index set.
    """

    def __init__(self, spec: Spec):
        self.spec = spec
        B = spec.batch
        if spec.ctx_log_uniform is not None:
            lo, hi = spec.ctx_log_uniform
            u = np.array([_rng(spec, r, 0, 0, _P_CTX).random() for r in range(B)])
            self.ctx = np.rint(np.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))).astype(np.int64)
        else:
            self.ctx = np.full(B, spec.ctx, dtype=np.int64)
        if spec.retention_range is not None:
            lo, hi = spec.retention_range
            self.p = np.array([lo + (hi - lo) * _rng(spec, r, 0, 0, _P_RET).random() for r in range(B)])
        else:
            self.p = np.full(B, spec.retention, dtype=np.float64)
        extra = spec.topk - int(round(spec.overlap * spec.topk)) if spec.n_q > 1 else 0
        if np.any(self.ctx < spec.topk + extra):
            raise ValueError("context shorter than the selection")
        self._prev = [None] * B   # token-0 selection (non-window part) of the last step
        self._next_t = 0
        self._hot = None          # controlled-reuse mode: hot set and fresh stream per request
        self._fresh = None
        if spec.mode == "zipf_window":
            # base verified length: the last step's speculative tokens end at ctx
            self._n0 = int(spec.ctx) - spec.n_q + 1 - (spec.steps - 1)
            if self._n0 - spec.window < spec.topk:
                raise ValueError("context too short for the recency window")
            self._zmod = 1 << int(math.ceil(math.log2(spec.ctx)))
            self._zmul = np.empty(B, dtype=np.int64)
            self._zoff = np.empty(B, dtype=np.int64)
            for r in range(B):
                g = _rng(spec, r, 0, 0, _P_ZMAP)
                self._zmul[r] = int(g.integers(0, self._zmod // 2)) * 2 + 1
                self._zoff[r] = int(g.integers(0, self._zmod))

    # ---- verified context length (speculative positions start here) ----
    def verified_len(self, t: int) -> np.ndarray:
        s = self.spec
        if s.mode == "zipf_window":
            return np.full(s.batch, self._n0 + t, dtype=np.int64)
        return self.ctx.copy()

    def speculative_rows(self, t: int):
        """(first_row, n_rows) of the positions whose host rows are rewritten
        before step t (draft tokens of this step), or None."""
        s = self.spec
        if not s.speculative:
            return None
        return (self._n0 + t, s.n_q - 1)

    # ---- hot-token (Zipf) draws for the stress mix ----
    def _zipf_draw(self, rng, r: int, need: int, limit: int, exclude: np.ndarray) -> np.ndarray:
        out = np.empty(0, dtype=np.int64)
        excl = np.asarray(exclude, dtype=np.int64)
        guard = 0
        while out.size < need:
            guard += 1
            if guard > 10000:
                raise RuntimeError("zipf draw did not converge")
            rank = rng.zipf(self.spec.zipf_s, size=max(4 * (need - out.size), 256)).astype(np.int64)
            rank = rank[(rank >= 1) & (rank <= self._zmod)]
            pos = ((rank - 1) * self._zmul[r] + self._zoff[r]) % self._zmod
            pos = pos[pos < limit]
            _, first = np.unique(pos, return_index=True)
            pos = pos[np.sort(first)]
            pos = pos[~np.isin(pos, excl)]
            pos = pos[~np.isin(pos, out)]
            out = np.concatenate([out, pos[: need - out.size]])
        return out

    def _controlled_step(self, r: int, t: int) -> np.ndarray:
        """Controlled reuse: a fixed hot set of round(p*K) ids is selected at
        every step and the remaining ids are fresh (never selected before by
        this request), so once the hot set is resident the adjacent-step
        reuse is p."""
        s = self.spec
        K, ctx = s.topk, int(self.ctx[r])
        if self._hot is None:
            self._hot = [None] * s.batch
            self._fresh = [None] * s.batch
        if self._hot[r] is None:
            g = _rng(s, r, 0, 0, _P_INIT)
            n_hot = int(round(self.p[r] * K))
            perm = g.permutation(ctx).astype(np.int64)
            self._hot[r] = perm[:n_hot]
            self._fresh[r] = perm[n_hot:]
        hot = self._hot[r]
        m = K - hot.size
        if (t + 1) * m > self._fresh[r].size:
            raise ValueError("context too short for this many fresh selections")
        fresh = self._fresh[r][t * m:(t + 1) * m]
        sel = _rng(s, r, t, 0, _P_PERM).permutation(np.concatenate([hot, fresh]))
        return np.tile(sel, (s.n_q, 1))

    def _request_step(self, r: int, t: int) -> np.ndarray:
        s = self.spec
        if s.mode == "controlled":
            return self._controlled_step(r, t)
        K, ctx = s.topk, int(self.ctx[r])
        out = np.empty((s.n_q, K), dtype=np.int64)
        if s.mode == "uniform":
            if t == 0:
                base = _rng(s, r, t, 0, _P_INIT).choice(ctx, size=K, replace=False).astype(np.int64)
            else:
                prev = self._prev[r]
                keep = _rng(s, r, t, 0, _P_KEEP).random(K) < self.p[r]
                kept = prev[keep]
                new = _draw_excluding(_rng(s, r, t, 0, _P_REDRAW), 0, ctx, K - kept.size, kept)
                base = np.concatenate([kept, new])
            base = _rng(s, r, t, 0, _P_PERM).permutation(base)
            self._prev[r] = base
            out[0] = base
            for g in range(1, s.n_q):
                rg = _rng(s, r, t, g, _P_TOKEN)
                n_keep = int(round(s.overlap * K))
                shared = base[np.sort(rg.choice(K, size=n_keep, replace=False))]
                extra = _draw_excluding(rg, 0, ctx, K - n_keep, base)
                out[g] = rg.permutation(np.concatenate([shared, extra]))
            return out
        # zipf_window: recency window + Zipf hot set with retention
        W = s.window
        M = K - W
        n_t = self._n0 + t
        limit = self._n0 - W   # every non-window position stays verified and off-window
        if t == 0:
            hot = self._zipf_draw(_rng(s, r, t, 0, _P_INIT), r, M, limit, np.empty(0, np.int64))
        else:
            prev = self._prev[r]
            keep = _rng(s, r, t, 0, _P_KEEP).random(M) < self.p[r]
            kept = prev[keep]
            new = self._zipf_draw(_rng(s, r, t, 0, _P_REDRAW), r, M - kept.size, limit, kept)
            hot = np.concatenate([kept, new])
        self._prev[r] = hot
        for g in range(s.n_q):
            win = np.arange(n_t + g - W, n_t + g, dtype=np.int64)
            if g == 0:
                sel = hot
            else:
                rg = _rng(s, r, t, g, _P_TOKEN)
                n_keep = int(round(s.overlap * M))
                shared = hot[np.sort(rg.choice(M, size=n_keep, replace=False))]
                extra = self._zipf_draw(rg, r, M - n_keep, limit, hot)
                sel = np.concatenate([shared, extra])
            out[g] = _rng(s, r, t, g, _P_PERM).permutation(np.concatenate([win, sel]))
        return out

    def topk(self, t: int) -> np.ndarray:
        """X for step t as int32 [B][n_q][K]; steps must be taken in order."""
        if t != self._next_t:
            raise ValueError(f"steps must be generated in order (expected {self._next_t}, got {t})")
        if self.spec.mode == "zipf_window" and t >= self.spec.steps:
            raise ValueError("the stress mix is defined for its own step count only")
        X = np.stack([self._request_step(r, t) for r in range(self.spec.batch)])
        self._next_t += 1
        return X.astype(np.int32)

    def all_steps(self, n: int) -> np.ndarray:
        return np.stack([self.topk(t) for t in range(n)])

    # ---- host rows ----
    def host_rows_total(self) -> int:
        return int(self.ctx.sum())

    def request_row_offsets(self) -> np.ndarray:
        """Row offset of each request inside one contiguous host region."""
        return np.concatenate([[0], np.cumsum(self.ctx)[:-1]]).astype(np.int64)


# ---------------------------------------------------------------------------
# native filler for host rows
# ---------------------------------------------------------------------------
def build(force: bool = True) -> str:
    """Compile fill.c into libavsg_workload.so (gcc, OpenMP)."""
    src = os.path.join(_HERE, "fill.c")
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(src):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-shared", "-fPIC", "-std=c11",
                               "-o", tmp, src])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        lib.avsg_wl_fill_rows.restype = ctypes.c_int
        lib.avsg_wl_fill_rows.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int, ctypes.c_uint64, ctypes.c_int]
        lib.avsg_wl_key.restype = ctypes.c_uint64
        lib.avsg_wl_key.argtypes = [ctypes.c_uint64] * 5
        _lib = lib
    return _lib


def default_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def row_key(spec: Spec, stream: int, request: int, version: int = 0) -> int:
    return int(_load().avsg_wl_key(spec.seed, spec.cfg_id, stream, request, version))


def fill_rows(ptr: int, first_row: int, n_rows: int, row_bytes: int, kind: int, key: int,
              nthreads: Optional[int] = None) -> None:
    """Write seeded contents into rows [first_row, first_row + n_rows) of the
    region at address `ptr` (row 0 at ptr)."""
    rc = _load().avsg_wl_fill_rows(ctypes.c_void_p(ptr), first_row, n_rows, row_bytes, kind,
                                   ctypes.c_uint64(key), nthreads or default_threads())
    if rc != 0:
        raise ValueError("avsg_wl_fill_rows: bad arguments")


def stream_kind(stream: int) -> int:
    return 0 if stream == 0 else 1


def fill_host(wl: Workload, stream: int, ptr: int, version_rows=None,
              nthreads: Optional[int] = None) -> None:
    """Fill one stream's host region (all requests, contiguous) at `ptr`."""
    spec = wl.spec
    rb = spec.row_bytes[stream]
    offs = wl.request_row_offsets()
    for r in range(spec.batch):
        fill_rows(ptr + int(offs[r]) * rb, 0, int(wl.ctx[r]), rb, stream_kind(stream),
                  row_key(spec, stream, r, 0), nthreads)


def refresh_speculative(wl: Workload, t: int, stream_ptrs: Sequence[int],
                        nthreads: Optional[int] = None) -> None:
    """Rewrite the draft-token rows used by step t (new content per step),
    as a serving engine would after regenerating rejected speculative KV."""
    sr = wl.speculative_rows(t)
    if sr is None:
        return
    first, n = sr
    spec = wl.spec
    offs = wl.request_row_offsets()
    for s, ptr in enumerate(stream_ptrs):
        rb = spec.row_bytes[s]
        for r in range(spec.batch):
            fill_rows(ptr + int(offs[r]) * rb, first, n, rb, stream_kind(s),
                      row_key(spec, s, r, t + 1), nthreads)
