"""The C-ABI library loads and exports every entry point include/avsg.h declares,
and host-side validation behaves as documented (no GPU needed)."""
import ctypes
import os
import re

import pytest

import paper_2609_37538_amd.avsg as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "avsg.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(avsg_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(A.LIB_PATH):
        from paper_2609_37538_amd import _build
        _build.build()
    return A.load()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(lib, n), f"{n} declared in avsg.h but not exported"


def test_binding_has_same_names(lib):
    for n in declared_functions():
        assert hasattr(A, n), f"binding lacks {n}"


def test_struct_layouts_match_header(lib, tmp_path):
    """Every field offset and the size of the binding's structs equal what a C
    compiler makes of include/avsg.h."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "avsg.h"', "int main(void) {"]
    for cname, py in (("avsg_config", A.AvsgConfig), ("avsg_stats_t", A.AvsgStats)):
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l}
    for cname, py in (("avsg_config", A.AvsgConfig), ("avsg_stats_t", A.AvsgStats)):
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, f"{cname}.{fname}"


def test_strerror(lib):
    assert A.avsg_strerror(0) == "ok"
    assert "capacity" in A.avsg_strerror(A.AVSG_E_CAPACITY)
    assert A.avsg_strerror(12345) == "unknown status"


def ws(**kw):
    base = dict(batch=64, topk=2048, n_q=2, slots=8192, row_bytes=(1152, 132))
    base.update(kw)
    return A.avsg_workspace_bytes(A.make_config(**base))


def test_check_config_statuses(lib):
    def chk(**kw):
        base = dict(batch=64, topk=2048, n_q=2, slots=8192, row_bytes=(1152, 132))
        base.update(kw)
        return A.avsg_check_config(A.make_config(**base))
    assert chk() == A.AVSG_OK
    assert chk(slots=12288) == A.AVSG_E_NOTPOW2
    assert chk(slots=2048) == A.AVSG_E_CAPACITY
    assert chk(slots=32768, n_q=1) == A.AVSG_E_CAPACITY      # beyond one workgroup's LDS
    assert chk(slots=16384, topk=1024) == A.AVSG_OK           # 9*16384 + 12*1024 bytes fit
    assert chk(slots=16384, topk=2048) == A.AVSG_E_CAPACITY
    assert chk(max_life=0) == A.AVSG_E_RANGE
    assert chk(batch=0) == A.AVSG_E_INVAL
    assert chk(match_mode=A.AVSG_MATCH_DUALPTR) == A.AVSG_E_UNSUPPORTED
    # resident reuse: hash matching only; its index map must fit beside the table
    assert chk(gather_mode=A.AVSG_GATHER_RESIDENT) == A.AVSG_OK
    assert chk(n_q=1, slots=2048, match_mode=A.AVSG_MATCH_DUALPTR,
               gather_mode=A.AVSG_GATHER_RESIDENT) == A.AVSG_E_UNSUPPORTED
    assert chk(batch=1, topk=128, n_q=62, slots=16384, gather_mode=A.AVSG_GATHER_RESIDENT) == A.AVSG_OK
    assert chk(batch=1, topk=128, n_q=63, slots=16384, gather_mode=A.AVSG_GATHER_RESIDENT) == \
        A.AVSG_E_CAPACITY
    assert chk(batch=1, topk=128, n_q=110, slots=16384) == A.AVSG_OK
    assert chk(gather_mode=9) == A.AVSG_E_INVAL
    # early fetch: hash matching only; knobs 0 / -1
    assert chk(gather_mode=A.AVSG_GATHER_EARLY) == A.AVSG_OK
    assert chk(gather_mode=A.AVSG_GATHER_EARLY, early_staging_rows=-1, early_direct=-1) == A.AVSG_OK
    assert chk(gather_mode=A.AVSG_GATHER_EARLY, early_staging_rows=-2) == A.AVSG_E_INVAL
    assert chk(gather_mode=A.AVSG_GATHER_EARLY, early_direct=1) == A.AVSG_E_INVAL
    assert chk(n_q=1, slots=2048, match_mode=A.AVSG_MATCH_DUALPTR,
               gather_mode=A.AVSG_GATHER_EARLY) == A.AVSG_E_UNSUPPORTED
    assert chk(batch=1, topk=128, n_q=62, slots=16384, gather_mode=A.AVSG_GATHER_EARLY) == A.AVSG_OK


def test_workspace_size_and_validation(lib):
    n = ws()
    B, S, K, nq = 64, 8192, 2048, 2
    assert n >= 8 * B * S + 8 * B * nq * K
    assert n % 256 == 0
    assert ws(slots=12288) == 0                 # not a power of two
    assert ws(slots=2048) == 0                  # S < N_q K (Eq. 7)
    assert ws(max_life=0) == 0 and ws(max_life=128) == 0
    assert ws(a1=7, a2=7) == 0                  # primes must differ
    assert ws(a1=9) == 0                        # 9 is not prime
    assert ws(retry=-1) == 0
    assert ws(row_bytes=(1150,)) == 0           # not a multiple of 4
    assert ws(batch=0) == 0 and ws(batch=1025) == 0
    assert ws(topk=8192, n_q=1, slots=8192) == 0   # beyond 4096 indices per token
    assert ws(match_mode=A.AVSG_MATCH_DUALPTR, n_q=1, slots=2048) > 0
    assert ws(match_mode=A.AVSG_MATCH_DUALPTR, n_q=2) == 0
    assert ws(gather_mode=9) == 0
    assert ws(gather_mode=A.AVSG_GATHER_AUTO) == ws(gather_mode=A.AVSG_GATHER_RESIDENT)
    # the resident-reuse plan adds three transfer lists, fan slots, counts and claims
    B, nq, K = 64, 2, 2048
    assert ws(gather_mode=A.AVSG_GATHER_RESIDENT) >= ws() + (3 * 8 + 4) * B * nq * K + 12 * B
    assert ws(gather_mode=A.AVSG_GATHER_POSITION) > ws() - 1
    # early fetch adds keys, positions, finish entries and 16384 staging rows of both streams
    early = ws(gather_mode=A.AVSG_GATHER_EARLY)
    assert early >= ws(gather_mode=A.AVSG_GATHER_RESIDENT) + 36 * B * nq * K + 16384 * (1152 + 132)
    assert ws(gather_mode=A.AVSG_GATHER_EARLY, early_staging_rows=-1) == early - 16384 * (1152 + 132)
    assert ws(match_mode=A.AVSG_MATCH_DUALPTR, n_q=1, slots=2048, gather_mode=A.AVSG_GATHER_POSITION) == 0
    assert ws(n_q=1, slots=2, topk=1, batch=1, row_bytes=(4,)) > 0
    assert ws(n_q=127, topk=64, slots=8192, row_bytes=(4,)) > 0
    assert ws(n_q=128, topk=64, slots=8192, row_bytes=(4,)) == 0


def test_auto_transfer_resolution(lib):
    """AVSG_GATHER_AUTO: resident reuse from 8192 lookups per step (B * N_q * K)
    with hash matching when its plan fits, else the paper's S3; the workspace
    is the chosen transfer's."""
    def res(**kw):
        base = dict(row_bytes=(1152,), gather_mode=A.AVSG_GATHER_AUTO)
        base.update(kw)
        cfg = A.make_config(**base)
        return A.avsg_resolve_config(cfg).gather_mode, A.avsg_workspace_bytes(cfg)
    def ws_of(mode, **kw):
        return A.avsg_workspace_bytes(A.make_config(row_bytes=(1152,), gather_mode=mode, **kw))
    tiny = dict(batch=1, topk=256, n_q=1, slots=1024)
    assert res(**tiny) == (A.AVSG_GATHER_BALANCED, ws_of(A.AVSG_GATHER_BALANCED, **tiny))
    b16 = dict(batch=16, topk=2048, n_q=1, slots=8192)
    assert res(**b16) == (A.AVSG_GATHER_RESIDENT, ws_of(A.AVSG_GATHER_RESIDENT, **b16))
    assert res(batch=2, topk=2048, n_q=1, slots=8192)[0] == A.AVSG_GATHER_BALANCED    # 4096 lookups
    assert res(batch=2, topk=2048, n_q=2, slots=8192)[0] == A.AVSG_GATHER_RESIDENT    # 8192 lookups
    assert res(batch=4, topk=2048, n_q=1, slots=2048,
               match_mode=A.AVSG_MATCH_DUALPTR)[0] == A.AVSG_GATHER_BALANCED
    # the resident plan would not fit beside this table: S3
    assert res(batch=1, topk=128, n_q=64, slots=16384)[0] == A.AVSG_GATHER_BALANCED
    # errors are those of the configuration itself
    assert A.avsg_check_config(A.make_config(batch=0, topk=64, n_q=1, slots=256,
                                             gather_mode=A.AVSG_GATHER_AUTO)) == A.AVSG_E_INVAL
    assert A.avsg_check_config(A.make_config(batch=1, topk=64, n_q=1, slots=96,
                                             gather_mode=A.AVSG_GATHER_AUTO)) == A.AVSG_E_NOTPOW2
    assert A.avsg_check_config(A.make_config(batch=1, topk=64, n_q=1, slots=256, gather_mode=9)) == A.AVSG_E_INVAL
