"""CPU oracle of the AVSG per-decode-step operator (test infrastructure only).

The method's oracle is plain C (``avsg_oracle.c``), compiled with gcc into
``liboracle_avsg.so`` and driven through ctypes with NumPy arrays;
``transfer_plan`` (plain Python) defines which misses the resident-reuse
transfer may fill from another slot, and ``early_set`` / ``transfer_plan_early``
which rows the early-fetch transfer may read from the host before Stage One
and what is left to plan after it.  Only the test suite, the smoke check and
the benchmark's CPU-baseline leg use this package; the product path never
imports it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle_avsg.so")
_SRC = os.path.join(_HERE, "avsg_oracle.c")

# Default probe primes (two distinct primes, Section 3.2).
A1_DEFAULT = 2654435761
A2_DEFAULT = 2246822519


ASAN_LIB_PATH = os.path.join(_HERE, "liboracle_avsg_asan.so")


def build(force: bool = True, sanitize: bool = False, native: bool = False, out: Optional[str] = None) -> str:
    """Compile the oracle with gcc (-O3, OpenMP over requests).  sanitize:
    AddressSanitizer + UndefinedBehaviorSanitizer build (-O1) for the
    sanitizer test; native: -march=native for the host it is built on (the
    benchmark builds that on the machine it times)."""
    if out is None:
        out = ASAN_LIB_PATH if sanitize else LIB_PATH
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(_SRC):
        flags = ["-O3", "-fopenmp", "-shared", "-fPIC", "-std=c11", "-Wall", "-Wextra"]
        if native:
            flags.append("-march=native")
        if sanitize:
            flags += ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                      "-fno-omit-frame-pointer", "-O1"]
        tmp = out + ".tmp"
        subprocess.check_call(["gcc", *flags, "-o", tmp, _SRC])
        os.replace(tmp, out)
    return out


class _Cfg(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("topk", ctypes.c_int32), ("n_q", ctypes.c_int32),
                ("slots", ctypes.c_int32), ("retry", ctypes.c_int32), ("max_life", ctypes.c_int32),
                ("a1", ctypes.c_uint32), ("a2", ctypes.c_uint32)]


class RefStats(ctypes.Structure):
    _fields_ = [("hits", ctypes.c_uint64), ("misses", ctypes.c_uint64),
                ("lost_exhausted", ctypes.c_uint64), ("lost_collision", ctypes.c_uint64),
                ("alloc_decays", ctypes.c_uint64), ("revivals", ctypes.c_uint64),
                ("invalidations", ctypes.c_uint64), ("max_step_alloc_decays", ctypes.c_int32),
                ("pad", ctypes.c_int32)]

    def as_dict(self):
        return {f: int(getattr(self, f)) for f, _ in self._fields_ if f != "pad"}


_lib = None
_P = ctypes.c_void_p


def _load():
    global _lib
    if _lib is None:
        # AVSG_ORACLE_LIB names another build of the same source (the
        # sanitizer test's, or the benchmark's -march=native build)
        path = os.environ.get("AVSG_ORACLE_LIB") or LIB_PATH
        if path == LIB_PATH and not os.path.exists(LIB_PATH):
            build(force=False)
        lib = ctypes.CDLL(path)
        lib.avsg_ref_create.restype = _P
        lib.avsg_ref_create.argtypes = [ctypes.POINTER(_Cfg), ctypes.POINTER(ctypes.c_int32)]
        lib.avsg_ref_destroy.argtypes = [_P]
        lib.avsg_ref_step.restype = ctypes.c_int32
        lib.avsg_ref_step.argtypes = [_P, _P, _P, _P, _P, _P, _P, ctypes.c_int32, _P, _P, _P, _P,
                                      ctypes.c_int32]
        lib.avsg_ref_export.argtypes = [_P, ctypes.c_int32, _P, _P]
        lib.avsg_ref_import.argtypes = [_P, ctypes.c_int32, _P, _P]
        lib.avsg_ref_stats.argtypes = [_P, ctypes.c_int32, ctypes.POINTER(RefStats)]
        lib.avsg_ref_pack.restype = ctypes.c_uint32
        lib.avsg_ref_pack.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_int64, ctypes.c_int64]
        lib.avsg_ref_decode.argtypes = [ctypes.c_int32, ctypes.c_uint32, _P, _P, _P, _P]
        lib.avsg_ref_phi.restype = ctypes.c_int64
        lib.avsg_ref_phi.argtypes = [ctypes.c_int32, ctypes.c_int64]
        lib.avsg_ref_probe.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, _P, _P]
        lib.avsg_ref_dp_create.restype = _P
        lib.avsg_ref_dp_create.argtypes = [ctypes.c_int32, ctypes.c_int32]
        lib.avsg_ref_dp_destroy.argtypes = [_P]
        lib.avsg_ref_dp_step.restype = ctypes.c_int32
        lib.avsg_ref_dp_step.argtypes = [_P, _P, _P, _P, _P, _P, ctypes.c_int32, _P, _P, _P,
                                         ctypes.c_int32]
        lib.avsg_ref_dp_export.argtypes = [_P, ctypes.c_int32, _P]
        lib.avsg_ref_partition_balanced.argtypes = [ctypes.c_int64, ctypes.c_int32, _P]
        lib.avsg_ref_partition_request.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                   ctypes.c_int32, _P]
        lib.avsg_ref_partition_position.argtypes = [ctypes.c_int64, ctypes.c_int32, _P]
        lib.avsg_ref_validate.argtypes = [_P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, _P]
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _ptr_array(ptrs: Sequence[int]):
    arr = (ctypes.c_void_p * len(ptrs))(*[ctypes.c_void_p(int(p)) for p in ptrs])
    return arr


def affinity_cpus() -> int:
    """CPUs this process may run on."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def thread_cap() -> int:
    """Upper bound on oracle threads: OMP_NUM_THREADS when set (the GPU
    machines set it to the CPU share of one GPU), else 16."""
    try:
        v = int(os.environ.get("OMP_NUM_THREADS", "0"))
    except ValueError:
        v = 0
    return v if v > 0 else 16


def default_threads() -> int:
    return max(1, min(affinity_cpus(), thread_cap()))


class OracleError(RuntimeError):
    pass


class Oracle:
    """Stateful CPU reference: one Hash-State table per request."""

    def __init__(self, batch, topk, n_q, slots, retry=3, max_life=16, a1=A1_DEFAULT,
                 a2=A2_DEFAULT, nthreads: Optional[int] = None):
        self.lib = _load()
        self.cfg = _Cfg(batch, topk, n_q, slots, retry, max_life, a1, a2)
        st = ctypes.c_int32(0)
        self.h = self.lib.avsg_ref_create(ctypes.byref(self.cfg), ctypes.byref(st))
        if not self.h:
            raise OracleError(f"avsg_ref_create failed with status {st.value}")
        self.B, self.K, self.n_q, self.S = batch, topk, n_q, slots
        self.nthreads = nthreads or default_threads()
        self.miss_x = np.zeros((batch, n_q * topk), dtype=np.int32)
        self.miss_o = np.zeros((batch, n_q * topk), dtype=np.int32)

    @staticmethod
    def create_status(batch, topk, n_q, slots, retry=3, max_life=16, a1=A1_DEFAULT,
                      a2=A2_DEFAULT) -> int:
        lib = _load()
        cfg = _Cfg(batch, topk, n_q, slots, retry, max_life, a1, a2)
        st = ctypes.c_int32(0)
        h = lib.avsg_ref_create(ctypes.byref(cfg), ctypes.byref(st))
        if h:
            lib.avsg_ref_destroy(h)
        return st.value

    def close(self):
        if self.h:
            self.lib.avsg_ref_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, X: np.ndarray, verified: Optional[np.ndarray] = None, host=None, buf=None,
             row_bytes=None, rows: Optional[np.ndarray] = None):
        """Run one decode step.  host/buf: lists of per-(stream, request)
        addresses ordered s*B + r; row_bytes: per stream.
        Returns (O [B][n_q][K], n [B][n_q]); the transfer lists are in
        self.miss_x / self.miss_o."""
        X = np.ascontiguousarray(X, dtype=np.int32)
        assert X.shape == (self.B, self.n_q, self.K), X.shape
        O = np.empty_like(X)
        n = np.empty((self.B, self.n_q), dtype=np.int32)
        ver = None if verified is None else np.ascontiguousarray(verified, dtype=np.int64)
        rws = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
        ns = 0
        hp = bp = rbp = None
        if host is not None:
            ns = len(row_bytes)
            hp = _ptr_array(host)
            bp = _ptr_array(buf)
            rb = np.ascontiguousarray(row_bytes, dtype=np.int64)
            rbp = _ptr(rb)
        rc = self.lib.avsg_ref_step(self.h, _ptr(X), _ptr(ver), _ptr(O), _ptr(n),
                                    _ptr(self.miss_x), _ptr(self.miss_o), ns, hp, bp, rbp,
                                    _ptr(rws), self.nthreads)
        if rc != 0:
            raise OracleError(f"avsg_ref_step returned {rc}")
        return O, n

    def misses(self, r: int, n_r: np.ndarray):
        tot = int(np.sum(n_r))
        return self.miss_x[r, :tot].copy(), self.miss_o[r, :tot].copy()

    def export(self, r: int):
        c = np.empty(self.S, dtype=np.int32)
        q = np.empty(self.S, dtype=np.uint32)
        self.lib.avsg_ref_export(self.h, r, _ptr(c), _ptr(q))
        return c, q

    def import_table(self, r: int, c: np.ndarray, q: np.ndarray):
        c = np.ascontiguousarray(c, dtype=np.int32)
        q = np.ascontiguousarray(q, dtype=np.uint32)
        assert c.shape == (self.S,) and q.shape == (self.S,)
        self.lib.avsg_ref_import(self.h, r, _ptr(c), _ptr(q))

    def stats(self, r: int) -> dict:
        s = RefStats()
        self.lib.avsg_ref_stats(self.h, r, ctypes.byref(s))
        return s.as_dict()

    def total_stats(self) -> dict:
        tot = {}
        for r in range(self.B):
            for k, v in self.stats(r).items():
                if k == "max_step_alloc_decays":
                    tot[k] = max(tot.get(k, 0), v)
                else:
                    tot[k] = tot.get(k, 0) + v
        return tot

    def probe(self, r: int, x: int):
        hit = ctypes.c_int32(0)
        h = ctypes.c_int32(0)
        self.lib.avsg_ref_probe(self.h, r, x, ctypes.byref(hit), ctypes.byref(h))
        return bool(hit.value), h.value


class DualPointerOracle:
    """Scalar sort-merge matching baseline with an S = K buffer."""

    def __init__(self, batch, topk, nthreads: Optional[int] = None):
        self.lib = _load()
        self.h = self.lib.avsg_ref_dp_create(batch, topk)
        if not self.h:
            raise OracleError("avsg_ref_dp_create failed")
        self.B, self.K = batch, topk
        self.nthreads = nthreads or default_threads()
        self.miss_x = np.zeros((batch, topk), dtype=np.int32)
        self.miss_o = np.zeros((batch, topk), dtype=np.int32)

    def close(self):
        if self.h:
            self.lib.avsg_ref_dp_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, X: np.ndarray, host=None, buf=None, row_bytes=None):
        X = np.ascontiguousarray(X, dtype=np.int32).reshape(self.B, 1, self.K)
        O = np.empty_like(X)
        n = np.empty((self.B, 1), dtype=np.int32)
        ns = 0
        hp = bp = rbp = None
        if host is not None:
            ns = len(row_bytes)
            hp, bp = _ptr_array(host), _ptr_array(buf)
            rb = np.ascontiguousarray(row_bytes, dtype=np.int64)
            rbp = _ptr(rb)
        self.lib.avsg_ref_dp_step(self.h, _ptr(X), _ptr(O), _ptr(n), _ptr(self.miss_x),
                                  _ptr(self.miss_o), ns, hp, bp, rbp, self.nthreads)
        return O, n

    def export(self, r: int):
        c = np.empty(self.K, dtype=np.int32)
        self.lib.avsg_ref_dp_export(self.h, r, _ptr(c))
        return c


def pack(m, lifetime, invalid, fingerprint, slot) -> int:
    return int(_load().avsg_ref_pack(m, lifetime, invalid, fingerprint, slot))


def decode(m, q):
    l, b = ctypes.c_int32(), ctypes.c_int32()
    fp, o = ctypes.c_int64(), ctypes.c_int64()
    _load().avsg_ref_decode(m, ctypes.c_uint32(q), ctypes.byref(l), ctypes.byref(b),
                            ctypes.byref(fp), ctypes.byref(o))
    return l.value, b.value, fp.value, o.value


def phi(m, x) -> int:
    return int(_load().avsg_ref_phi(m, x))


def transfer_plan(miss_x, miss_o, c_after, rows_r: int):
    """Resident-reuse plan of one request-step: which misses must cross the host
    link.  This is a property of the transfer, not of the paper's method, whose
    Stage Two copies every miss from the host (Section 3.4); filling a slot from
    another slot that holds the same row leaves the buffer unchanged.

    Plain definition, for each miss (x, o) of the step's transfer list in order:
      - x outside [0, rows_r): a host entry (the copy skips it);
      - else, if some slot j outside this step's reservations caches x after the
        step (c_after[j] == x; invalidated entries are already -1), a resident
        copy j -> o from the largest such j (its row arrived in an earlier step);
      - else, if o is the largest slot this step reserved for x, a host entry;
      - else a repeat of that host entry.
    Each host entry also carries two fan slots: the two largest repeat
    destinations of its index, larger first (-1 where there are fewer), which
    the host copy writes too; the other repeats stay in the repeat list,
    copied from the host entry's slot.
    Each list keeps transfer-list order.  Returns
    (host_x, host_o, host_fan, res_src, res_dst, rep_src, rep_dst) as int32
    arrays, host_fan of shape (n_host, 2).
    """
    miss_x = [int(v) for v in miss_x]
    miss_o = [int(v) for v in miss_o]
    c_after = np.asarray(c_after)
    reserved = set(miss_o)
    wanted = {x for x in miss_x if 0 <= x < rows_r}
    resident = {}
    for j in range(len(c_after)):          # ascending, so the largest slot stays
        x = int(c_after[j])
        if x in wanted and j not in reserved:
            resident[x] = j
    first = {}
    for x, o in zip(miss_x, miss_o):
        if 0 <= x < rows_r:
            first[x] = max(first.get(x, -1), o)
    repeats = {}
    for x, o in zip(miss_x, miss_o):
        if 0 <= x < rows_r and x not in resident and first[x] != o:
            repeats.setdefault(x, []).append(o)
    fan = {x: sorted(v, reverse=True)[:2] for x, v in repeats.items()}
    lists = [[] for _ in range(7)]
    for x, o in zip(miss_x, miss_o):
        valid = 0 <= x < rows_r
        if valid and x in resident:
            lists[3].append(resident[x])
            lists[4].append(o)
        elif valid and first[x] != o:
            if o not in fan[x]:
                lists[5].append(first[x])
                lists[6].append(o)
        else:
            lists[0].append(x)
            lists[1].append(o)
            lists[2].append(((fan.get(x, []) if valid else []) + [-1, -1])[:2])
    out = [np.asarray(v, dtype=np.int32) for v in lists]
    out[2] = out[2].reshape(-1, 2)
    return tuple(out)


EARLY_MAX_POSITIONS = 4


def early_set(X_r, c_before, rows_r: int, max_positions: int = EARLY_MAX_POSITIONS):
    """Indices of one request-step whose rows can cross the host link before
    Stage One has run.  Like transfer_plan, a property of the transfer, not of
    the paper's method.

    Plain definition: the distinct indices x of the step's selections X_r
    (every token) such that
      - 0 <= x < rows_r,
      - c_before[j] != x for every slot j (no slot held x when the step began),
      - x occurs at most max_positions times over the step's tokens.
    Such an x misses where it first occurs (no slot can satisfy c[o] == x), and
    no slot outside the step's reservations caches it afterwards, so the
    paper's Stage Two reads its row from the host whatever the slots turn out
    to be; every position of x ends with x's row in its slot.
    Returns (keys ascending, positions): positions[k] lists the flat positions
    g * K + i of keys[k] in increasing order."""
    X_r = np.asarray(X_r).reshape(-1)
    cached = {int(v) for v in np.asarray(c_before).tolist()}
    where = {}
    for pos, x in enumerate(X_r.tolist()):
        if 0 <= x < rows_r:
            where.setdefault(int(x), []).append(pos)
    keys = sorted(x for x, p in where.items() if x not in cached and len(p) <= max_positions)
    return np.asarray(keys, dtype=np.int32), [where[x] for x in keys]


def transfer_plan_early(miss_x, miss_o, c_after, rows_r: int, early_keys):
    """Resident-reuse plan of the misses left to Stage Two once the early
    fetch (early_set) has written every position of its keys: transfer_plan
    over the transfer list without the misses of early keys.  Dropping them
    changes no other entry: an early key's slots cache that key (or nothing),
    so they are never a resident source of another index.
    Returns the seven lists of transfer_plan."""
    early = {int(v) for v in np.asarray(early_keys).tolist()}
    keep = [k for k, x in enumerate(np.asarray(miss_x).tolist()) if int(x) not in early]
    mx = np.asarray(miss_x, dtype=np.int32)[keep]
    mo = np.asarray(miss_o, dtype=np.int32)[keep]
    return transfer_plan(mx, mo, c_after, rows_r)


def validate(X: np.ndarray, rows) -> np.ndarray:
    """Per token row of X [B][n_q][K]: 1 if an index lies outside
    [0, rows[r]), plus 2 if an in-range index repeats in the row, else 0
    (the C oracle's avsg_ref_validate)."""
    X = np.ascontiguousarray(X, dtype=np.int32)
    B, n_q, K = X.shape
    rws = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty(B * n_q, dtype=np.int32)
    _load().avsg_ref_validate(_ptr(X), B, n_q, K, _ptr(rws), _ptr(out))
    return out.reshape(B, n_q)


def partition_balanced(n_miss: int, C: int) -> np.ndarray:
    out = np.empty(C + 1, dtype=np.int64)
    _load().avsg_ref_partition_balanced(n_miss, C, _ptr(out))
    return out


def partition_request(B: int, C: int, n_q: int, K: int) -> np.ndarray:
    out = np.empty(C, dtype=np.int64)
    _load().avsg_ref_partition_request(B, C, n_q, K, _ptr(out))
    return out


def partition_position(n_positions: int, C: int) -> np.ndarray:
    out = np.empty(C + 1, dtype=np.int64)
    _load().avsg_ref_partition_position(n_positions, C, _ptr(out))
    return out
