"""AVSG per-decode-step sparse-gather operator for MI355X (gfx950).

The operator lives in the HIP library ``libavsg.so`` (C ABI in
``include/avsg.h``); :mod:`paper_2609_37538_amd.avsg` is its ctypes binding.
"""
from .avsg import (  # noqa: F401
    AVSG_GATHER_BALANCED, AVSG_GATHER_NONE, AVSG_GATHER_PIPELINED, AVSG_GATHER_POSITION,
    AVSG_GATHER_REQUEST, AVSG_GATHER_RESIDENT,
    AVSG_GATHER_SDMA,
    AVSG_MATCH_DUALPTR, AVSG_MATCH_HASH, AvsgConfig, AvsgError, HostRegion, Operator,
    avsg_check_config, avsg_create, avsg_destroy, avsg_device_cus, avsg_export_misses, avsg_export_plan, avsg_export_state,
    avsg_h2d_peak, avsg_host_alloc, avsg_host_free, avsg_reset_request, avsg_reset_stats,
    avsg_set_timing, avsg_stats, avsg_step, avsg_strerror, avsg_timing, avsg_workspace_bytes,
    load, make_config,
)


def build(verbose: bool = False) -> str:
    from ._build import build as _b
    return _b(verbose=verbose)
