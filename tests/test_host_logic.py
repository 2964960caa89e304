"""Host-side logic that needs no GPU: the benchmark's refusal of several GPUs,
the committed counter summary it reads, the product package's independence
from the oracle, and the binding's loud failure without the HIP library."""
import ast
import json
import os
import re
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_37538_amd")


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def _bench():
    sys.path.insert(0, ROOT)
    import bench
    return bench


def _default_args(**kw):
    a = dict(config="batch64_mtp2", warmup=16, steps=240, workers=0, gather="resident", match="hash")
    a.update(kw)
    return types.SimpleNamespace(**a)


def test_traffic_summary_block_is_complete():
    """The counter summary bench.py reads holds every field it reports, and its
    traffic is FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0 bytes."""
    bench = _bench()
    text = open(os.path.join(ROOT, bench.TRAFFIC_SUMMARY)).read()
    m = re.search(r"```json\n(.*?)\n```", text, re.S)
    assert m, "no machine-readable block"
    b = json.loads(m.group(1))
    for k in ("kernel", "workload", "source_sha256_16", "fetch_size_kib_per_launch", "fetch_factor",
              "write_size_kib_per_launch", "write_factor", "traffic_bytes_per_launch",
              "algorithmic_host_bytes_per_launch"):
        assert k in b, k
    want = b["fetch_size_kib_per_launch"] * 1024 * b["fetch_factor"] + \
        b["write_size_kib_per_launch"] * 1024 * b["write_factor"]
    assert abs(b["traffic_bytes_per_launch"] - want) <= 2
    assert b["kernel"] == "gather_resident_kernel" and b["workload"] == "batch64_mtp2"


@pytest.mark.parametrize("change", [dict(config="batch16"), dict(workers=64), dict(gather="balanced"),
                                    dict(match="dualptr")])
def test_traffic_only_for_the_profiled_run(change):
    """Traffic is reported for the profiled workload and transfer only (the
    step counts do not matter: a launch's traffic changes little from step to
    step).  The current summary matches the current code."""
    args = _default_args(**change)
    assert _bench().measured_traffic(args, args.gather) is None
    assert _bench().measured_traffic(_default_args(steps=20, warmup=5), "resident") is not None


def test_traffic_follows_the_source_hash(tmp_path, monkeypatch):
    """A summary whose hash does not match the sources yields no traffic."""
    bench = _bench()
    text = open(os.path.join(ROOT, bench.TRAFFIC_SUMMARY)).read()
    stale = re.sub(r'"source_sha256_16": "[0-9a-f]+"', '"source_sha256_16": "0000000000000000"', text)
    (tmp_path / "profiles").mkdir()
    (tmp_path / bench.TRAFFIC_SUMMARY).write_text(stale)
    for p in bench.GATHER_SOURCES:
        dst = tmp_path / p
        dst.parent.mkdir(parents=True, exist_ok=True)
        dst.write_bytes(open(os.path.join(ROOT, p), "rb").read())
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.measured_traffic(_default_args(), "resident") is None


def _imports(path):
    tree = ast.parse(open(path).read())
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            for a in node.names:
                yield a.name
        elif isinstance(node, ast.ImportFrom):
            yield node.module or ""


def test_product_package_never_imports_the_oracle():
    for name in os.listdir(PKG):
        if name.endswith(".py"):
            for mod in _imports(os.path.join(PKG, name)):
                assert not mod.split(".")[0] == "oracle", f"{name} imports {mod}"


def test_product_sources_do_not_include_oracle_code():
    csrc = os.path.join(PKG, "csrc")
    for name in os.listdir(csrc):
        text = open(os.path.join(csrc, name), errors="replace").read()
        for inc in re.findall(r'#include\s+["<]([^">]+)', text):
            assert "oracle" not in inc, f"{name} includes {inc}"


def test_binding_fails_loudly_without_the_library(tmp_path):
    code = (
        "import paper_2609_37538_amd.avsg as A\n"
        f"A.LIB_PATH = {str(tmp_path / 'missing.so')!r}\n"
        "A._lib = None\n"
        "try:\n"
        "    A.load()\n"
        "except ImportError as e:\n"
        "    print('raised:', e)\n"
        "else:\n"
        "    print('loaded')\n")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("raised:") and "no other implementation" in r.stdout
