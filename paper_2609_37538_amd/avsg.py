"""ctypes binding of libavsg (include/avsg.h): the same entry points, argument
marshalling only.  Every step of the operator runs in the library's HIP
kernels; if the library is missing this module raises at import-use time
rather than falling back to anything else.

`Operator` is a convenience wrapper that allocates the device workspace, the
buffers and the step outputs as PyTorch tensors (PyTorch supplies device
memory and streams only).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libavsg.so")

AVSG_OK = 0
AVSG_E_INVAL = -1
AVSG_E_NOTPOW2 = -2
AVSG_E_CAPACITY = -3
AVSG_E_RANGE = -4
AVSG_E_BADINDEX = -5
AVSG_E_HIP = -6
AVSG_E_INTERNAL = -7
AVSG_E_UNSUPPORTED = -8

AVSG_MATCH_HASH = 0
AVSG_MATCH_DUALPTR = 1
AVSG_GATHER_BALANCED = 0
AVSG_GATHER_REQUEST = 1
AVSG_GATHER_SDMA = 2
AVSG_GATHER_NONE = 3
AVSG_GATHER_POSITION = 4
AVSG_GATHER_PIPELINED = 5
AVSG_GATHER_RESIDENT = 6
AVSG_GATHER_EARLY = 7
AVSG_GATHER_AUTO = 8
AVSG_MAX_STREAMS = 2

A1_DEFAULT = 2654435761
A2_DEFAULT = 2246822519


class AvsgConfig(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("topk", ctypes.c_int32), ("n_q", ctypes.c_int32),
        ("slots", ctypes.c_int32), ("retry", ctypes.c_int32), ("max_life", ctypes.c_int32),
        ("a1", ctypes.c_uint32), ("a2", ctypes.c_uint32),
        ("n_streams", ctypes.c_int32), ("gather_workers", ctypes.c_int32),
        ("row_bytes", ctypes.c_int64 * AVSG_MAX_STREAMS),
        ("match_mode", ctypes.c_int32), ("gather_mode", ctypes.c_int32),
        ("early_staging_rows", ctypes.c_int32), ("early_direct", ctypes.c_int32),
        ("validate", ctypes.c_int32),
    ]


class AvsgStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "steps", "lookups", "hits", "misses", "bytes_moved", "lost_exhausted", "lost_collision",
        "alloc_decays", "revivals", "invalidations", "bad_indices", "resident_rows",
        "duplicate_rows", "host_bytes")] + [
        ("max_step_alloc_decays", ctypes.c_int32), ("queue_timeouts", ctypes.c_int32),
        ("copy_calls", ctypes.c_uint64), ("early_rows", ctypes.c_uint64),
        ("early_staged_rows", ctypes.c_uint64), ("early_deferred_rows", ctypes.c_uint64)]

    def as_dict(self):
        return {f: int(getattr(self, f)) for f, _ in self._fields_}


class AvsgError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        msg = f"{where}: {strerror(status)} ({status})"
        if detail:
            msg += f": {detail}"
        super().__init__(msg)


_lib = None
_P = ctypes.c_void_p


def load(share_torch_runtime: bool = True):
    """Load libavsg.so; raises if it has not been built.  With
    share_torch_runtime (the default) torch is imported first when installed,
    so the library runs on torch's HIP runtime; a process that never uses
    torch passes False and gets the system runtime."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(the operator has no other implementation)")
    # PyTorch ships its own HIP runtime under the same soname as the system's;
    # whichever loads first serves the whole process, and torch cannot start
    # on a different one, so torch (when installed) goes first and the library
    # shares its runtime
    if share_torch_runtime:
        try:
            import torch  # noqa: F401
        except ImportError:
            pass
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    lib.avsg_check_config.restype = i32
    lib.avsg_check_config.argtypes = [ctypes.POINTER(AvsgConfig)]
    lib.avsg_resolve_config.restype = i32
    lib.avsg_resolve_config.argtypes = [ctypes.POINTER(AvsgConfig), ctypes.POINTER(AvsgConfig)]
    lib.avsg_workspace_bytes.restype = sz
    lib.avsg_workspace_bytes.argtypes = [ctypes.POINTER(AvsgConfig)]
    lib.avsg_create.restype = i32
    lib.avsg_create.argtypes = [ctypes.POINTER(AvsgConfig), _P, _P, _P, sz, _P, _P,
                                ctypes.POINTER(_P)]
    lib.avsg_step.restype = i32
    lib.avsg_step.argtypes = [_P, _P, _P, _P, _P, _P]
    lib.avsg_stats.restype = i32
    lib.avsg_stats.argtypes = [_P, ctypes.POINTER(AvsgStats)]
    lib.avsg_request_stats.restype = i32
    lib.avsg_request_stats.argtypes = [_P, i32, ctypes.POINTER(AvsgStats)]
    lib.avsg_reset_stats.restype = i32
    lib.avsg_reset_stats.argtypes = [_P, _P]
    lib.avsg_reset_request.restype = i32
    lib.avsg_reset_request.argtypes = [_P, i32, _P]
    lib.avsg_export_state.restype = i32
    lib.avsg_export_state.argtypes = [_P, i32, _P, _P]
    lib.avsg_import_state.restype = i32
    lib.avsg_import_state.argtypes = [_P, i32, _P, _P, _P]
    lib.avsg_export_misses.restype = i32
    lib.avsg_export_misses.argtypes = [_P, i32, _P, _P, _P]
    lib.avsg_export_plan.restype = i32
    lib.avsg_export_plan.argtypes = [_P, i32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
    lib.avsg_export_early.restype = i32
    lib.avsg_export_early.argtypes = [_P, i32, _P, _P, _P]
    lib.avsg_set_timing.restype = i32
    lib.avsg_set_timing.argtypes = [_P, i32]
    lib.avsg_timing.restype = i32
    lib.avsg_timing.argtypes = [_P, _P, _P, _P, i32, _P]
    lib.avsg_destroy.restype = i32
    lib.avsg_destroy.argtypes = [_P]
    lib.avsg_strerror.restype = ctypes.c_char_p
    lib.avsg_strerror.argtypes = [i32]
    lib.avsg_last_error.restype = ctypes.c_char_p
    lib.avsg_last_error.argtypes = [_P]
    lib.avsg_host_alloc.restype = i32
    lib.avsg_host_alloc.argtypes = [sz, i32, ctypes.POINTER(_P)]
    lib.avsg_host_free.restype = i32
    lib.avsg_host_free.argtypes = [_P]
    lib.avsg_h2d_peak.restype = i32
    lib.avsg_h2d_peak.argtypes = [_P, _P, sz, i32, _P, ctypes.POINTER(ctypes.c_double)]
    lib.avsg_device_cus.restype = i32
    lib.avsg_device_cus.argtypes = []
    lib.avsg_step_static.restype = i32
    lib.avsg_step_static.argtypes = [ctypes.POINTER(AvsgConfig), _P, _P, _P, _P, _P, _P, _P, i32, _P]
    _lib = lib
    return lib


def strerror(status: int) -> str:
    try:
        return load().avsg_strerror(status).decode()
    except ImportError:
        return "libavsg not built"


def _check(rc: int, where: str, h=None):
    if rc != AVSG_OK:
        detail = ""
        if h:
            detail = load().avsg_last_error(h).decode()
        raise AvsgError(rc, where, detail)


def _vp(x) -> Optional[ctypes.c_void_p]:
    return None if x is None or x == 0 else ctypes.c_void_p(int(x))


def _ptr_array(ptrs: Sequence[int]):
    return (ctypes.c_void_p * len(ptrs))(*[ctypes.c_void_p(int(p)) for p in ptrs])


def make_config(batch, topk, n_q, slots, retry=3, max_life=16, a1=A1_DEFAULT, a2=A2_DEFAULT,
                row_bytes=(1152,), gather_workers=0, match_mode=AVSG_MATCH_HASH,
                gather_mode=AVSG_GATHER_BALANCED, early_staging_rows=0, early_direct=0,
                validate=0) -> AvsgConfig:
    rb = (ctypes.c_int64 * AVSG_MAX_STREAMS)(*(list(row_bytes) + [0] * (AVSG_MAX_STREAMS - len(row_bytes))))
    return AvsgConfig(batch, topk, n_q, slots, retry, max_life, a1, a2, len(row_bytes),
                      gather_workers, rb, match_mode, gather_mode, early_staging_rows, early_direct,
                      validate)


# ---------------------------------------------------------------------------
# entry points, same names as the C ABI
# ---------------------------------------------------------------------------
def avsg_check_config(cfg: AvsgConfig) -> int:
    return int(load().avsg_check_config(ctypes.byref(cfg)))


def avsg_resolve_config(cfg: AvsgConfig) -> AvsgConfig:
    out = AvsgConfig()
    _check(load().avsg_resolve_config(ctypes.byref(cfg), ctypes.byref(out)), "avsg_resolve_config")
    return out


def avsg_workspace_bytes(cfg: AvsgConfig) -> int:
    return int(load().avsg_workspace_bytes(ctypes.byref(cfg)))


def avsg_create(cfg: AvsgConfig, host_rows: Sequence[int], rows_per_request, d_workspace: int,
                workspace_bytes: int, d_buffers: Sequence[int], stream: int = 0):
    rows = np.ascontiguousarray(rows_per_request, dtype=np.int64)
    h = ctypes.c_void_p()
    rc = load().avsg_create(ctypes.byref(cfg), _ptr_array(host_rows), rows.ctypes.data_as(_P),
                            _vp(d_workspace), workspace_bytes, _ptr_array(d_buffers), _vp(stream),
                            ctypes.byref(h))
    _check(rc, "avsg_create")
    return h


def avsg_step(h, d_topk: int, d_verified_len: Optional[int], d_slots: int, d_miss_counts: int,
              stream: int = 0) -> None:
    _check(load().avsg_step(h, _vp(d_topk), _vp(d_verified_len), _vp(d_slots), _vp(d_miss_counts),
                            _vp(stream)), "avsg_step", h)


def avsg_stats(h) -> dict:
    s = AvsgStats()
    _check(load().avsg_stats(h, ctypes.byref(s)), "avsg_stats", h)
    return s.as_dict()


def avsg_request_stats(h, r: int) -> dict:
    s = AvsgStats()
    _check(load().avsg_request_stats(h, r, ctypes.byref(s)), "avsg_request_stats", h)
    return s.as_dict()


def avsg_reset_stats(h, stream: int = 0) -> None:
    _check(load().avsg_reset_stats(h, _vp(stream)), "avsg_reset_stats", h)


def avsg_reset_request(h, r: int, stream: int = 0) -> None:
    _check(load().avsg_reset_request(h, r, _vp(stream)), "avsg_reset_request", h)


def avsg_export_state(h, r: int, slots: int):
    c = np.empty(slots, dtype=np.int32)
    q = np.empty(slots, dtype=np.uint32)
    _check(load().avsg_export_state(h, r, c.ctypes.data_as(_P), q.ctypes.data_as(_P)),
           "avsg_export_state", h)
    return c, q


def avsg_import_state(h, r: int, c, q, stream: int = 0) -> None:
    c = np.ascontiguousarray(c, dtype=np.int32)
    q = np.ascontiguousarray(q, dtype=np.uint32)
    _check(load().avsg_import_state(h, r, c.ctypes.data_as(_P), q.ctypes.data_as(_P), _vp(stream)),
           "avsg_import_state", h)


def avsg_export_plan(h, r: int, capacity: int):
    """(host_x, host_o, host_fan, res_src, res_dst, rep_src, rep_dst) of request
    r's last Stage Two plan; host_fan has two columns (the two fan slots of
    each host entry, -1 = none)."""
    n = [ctypes.c_int32(0) for _ in range(3)]
    a = [np.empty(2 * capacity if k == 2 else capacity, dtype=np.int32) for k in range(7)]
    P = [x.ctypes.data_as(_P) for x in a]
    _check(load().avsg_export_plan(h, r, ctypes.byref(n[0]), P[0], P[1], P[2], ctypes.byref(n[1]), P[3], P[4],
                                   ctypes.byref(n[2]), P[5], P[6]), "avsg_export_plan", h)
    sizes = [n[0].value] * 3 + [n[1].value] * 2 + [n[2].value] * 2
    out = [a[k][: sizes[k]].copy() for k in range(7)]
    out[2] = a[2][: 2 * sizes[2]].reshape(sizes[2], 2).copy()
    return tuple(out)


def avsg_export_misses(h, r: int, capacity: int):
    n = ctypes.c_int32(0)
    x = np.empty(capacity, dtype=np.int32)
    o = np.empty(capacity, dtype=np.int32)
    _check(load().avsg_export_misses(h, r, ctypes.byref(n), x.ctypes.data_as(_P),
                                     o.ctypes.data_as(_P)), "avsg_export_misses", h)
    return x[: n.value].copy(), o[: n.value].copy()


def avsg_export_early(h, r: int, capacity: int):
    """(keys, positions [n][4], -1 padded) of request r's last early list."""
    n = ctypes.c_int32(0)
    x = np.empty(capacity, dtype=np.int32)
    pos = np.empty((capacity, 4), dtype=np.int32)
    _check(load().avsg_export_early(h, r, ctypes.byref(n), x.ctypes.data_as(_P), pos.ctypes.data_as(_P)),
           "avsg_export_early", h)
    return x[: n.value].copy(), pos[: n.value].copy()


def avsg_set_timing(h, enable: bool) -> None:
    _check(load().avsg_set_timing(h, 1 if enable else 0), "avsg_set_timing", h)


def avsg_timing(h, cap: int):
    """(match_ms, gather_ms, tail_ms) per recorded step."""
    a = np.zeros(cap, dtype=np.float32)
    b = np.zeros(cap, dtype=np.float32)
    c = np.zeros(cap, dtype=np.float32)
    n = ctypes.c_int32(0)
    _check(load().avsg_timing(h, a.ctypes.data_as(_P), b.ctypes.data_as(_P), c.ctypes.data_as(_P), cap,
                              ctypes.byref(n)), "avsg_timing", h)
    return a[: n.value].copy(), b[: n.value].copy(), c[: n.value].copy()


def avsg_destroy(h) -> None:
    if h:
        _check(load().avsg_destroy(h), "avsg_destroy")


def avsg_strerror(status: int) -> str:
    return strerror(status)


def avsg_last_error(h) -> str:
    return load().avsg_last_error(h).decode() if h else ""


def avsg_host_alloc(nbytes: int, coherent: bool = False) -> int:
    p = ctypes.c_void_p()
    _check(load().avsg_host_alloc(nbytes, 1 if coherent else 0, ctypes.byref(p)), "avsg_host_alloc")
    return int(p.value)


def avsg_host_free(ptr: int) -> None:
    _check(load().avsg_host_free(_vp(ptr)), "avsg_host_free")


def avsg_h2d_peak(host: int, device: int, nbytes: int, iters: int = 20, stream: int = 0) -> float:
    g = ctypes.c_double(0.0)
    _check(load().avsg_h2d_peak(_vp(host), _vp(device), nbytes, iters, _vp(stream), ctypes.byref(g)),
           "avsg_h2d_peak")
    return float(g.value)


def avsg_device_cus() -> int:
    return int(load().avsg_device_cus())


def avsg_step_static(cfg: AvsgConfig, host_rows: Sequence[int], rows_per_request, d_buffers: Sequence[int],
                     d_topk: int, d_verified_len: Optional[int], d_slots: int, d_miss_counts: int,
                     cold_start: bool, stream: int = 0) -> None:
    rows = np.ascontiguousarray(rows_per_request, dtype=np.int64)
    _check(load().avsg_step_static(ctypes.byref(cfg), _ptr_array(host_rows), rows.ctypes.data_as(_P),
                                   _ptr_array(d_buffers), _vp(d_topk), _vp(d_verified_len), _vp(d_slots),
                                   _vp(d_miss_counts), 1 if cold_start else 0, _vp(stream)),
           "avsg_step_static")


# ---------------------------------------------------------------------------
# convenience wrappers (torch supplies device memory and streams)
# ---------------------------------------------------------------------------
class HostRegion:
    """Pinned, device-mapped host memory holding rows of one stream."""

    def __init__(self, nbytes: int, coherent: bool = False):
        self.nbytes = int(nbytes)
        self.ptr = avsg_host_alloc(self.nbytes, coherent)

    def view(self) -> np.ndarray:
        buf = (ctypes.c_uint8 * self.nbytes).from_address(self.ptr)
        return np.frombuffer(buf, dtype=np.uint8)

    def free(self):
        if self.ptr:
            avsg_host_free(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


class Operator:
    """One AVSG instance: config + workspace + buffers + outputs on cuda."""

    def __init__(self, cfg: AvsgConfig, host_rows: Sequence[int], rows_per_request, device=None,
                 stream=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        dev = torch.device(device or "cuda")
        self.device = dev
        self.stream = stream or torch.cuda.current_stream(dev)
        B, K, n_q, S = cfg.batch, cfg.topk, cfg.n_q, cfg.slots
        _check(avsg_check_config(cfg), "avsg_check_config")
        ws = avsg_workspace_bytes(cfg)
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=dev)
        self.buffers = [torch.zeros((B, S, int(cfg.row_bytes[s])), dtype=torch.uint8, device=dev)
                        for s in range(cfg.n_streams)]
        buf_ptrs = [self.buffers[s][r].data_ptr() for s in range(cfg.n_streams) for r in range(B)]
        self.slots = torch.empty((B, n_q, K), dtype=torch.int32, device=dev)
        self.miss_counts = torch.empty((B, n_q), dtype=torch.int32, device=dev)
        self.h = avsg_create(cfg, host_rows, rows_per_request, self.workspace.data_ptr(), ws, buf_ptrs,
                             self.stream.cuda_stream)

    def step(self, topk, verified_len=None):
        """topk: cuda int32 [B][n_q][K]; verified_len: cuda int64 [B] or None."""
        t = self.torch
        want = (self.cfg.batch, self.cfg.n_q, self.cfg.topk)
        if (topk.dtype != t.int32 or topk.device != self.slots.device or not topk.is_contiguous()
                or tuple(topk.shape) != want):
            raise ValueError(f"topk must be a contiguous int32 tensor of shape {want} on {self.slots.device}")
        vp = None
        if verified_len is not None:
            if (verified_len.dtype != t.int64 or verified_len.device != self.slots.device
                    or not verified_len.is_contiguous() or verified_len.numel() != self.cfg.batch):
                raise ValueError(f"verified_len must be a contiguous int64 tensor of {self.cfg.batch} "
                                 f"values on {self.slots.device}")
            vp = verified_len.data_ptr()
        avsg_step(self.h, topk.data_ptr(), vp, self.slots.data_ptr(), self.miss_counts.data_ptr(),
                  self.stream.cuda_stream)
        return self.slots, self.miss_counts

    def stats(self):
        return avsg_stats(self.h)

    def request_stats(self, r: int):
        return avsg_request_stats(self.h, r)

    def export_state(self, r: int):
        return avsg_export_state(self.h, r, self.cfg.slots)

    def export_misses(self, r: int):
        return avsg_export_misses(self.h, r, self.cfg.n_q * self.cfg.topk)

    def import_state(self, r: int, c, q):
        avsg_import_state(self.h, r, c, q, self.stream.cuda_stream)

    def export_plan(self, r: int):
        return avsg_export_plan(self.h, r, self.cfg.n_q * self.cfg.topk)

    def export_early(self, r: int):
        return avsg_export_early(self.h, r, self.cfg.n_q * self.cfg.topk)

    def close(self):
        if getattr(self, "h", None):
            avsg_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
