"""Host-side checks of bench.py (no GPU): the one-GPU contract and the
plumbing that attaches committed rocprofv3 traffic figures to the bench line."""
import importlib.util
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench_module():
    spec = importlib.util.spec_from_file_location("_bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_figures_follow_the_kernel_sources():
    b = _bench_module()
    rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    for sym, k in rec["kernels"].items():
        fam = sym.split("<")[0]
        if fam not in b.KERNEL_SOURCES:
            assert b.measured_traffic(sym) is None
            continue
        for f in b.KERNEL_SOURCES[fam]:
            assert os.path.exists(os.path.join(ROOT, "paper_2608_30877_amd", "csrc", f))
        # reported only while the sources hash to the profiled ones
        expect = int(k["bytes_per_launch"]) if k.get("source_sha256") == b.sources_sha256(fam) \
            else None
        assert b.measured_traffic(sym) == expect
    assert b.measured_traffic("no_such_kernel<0>") is None


def test_kernel_symbols_of_the_stack_projections():
    b = _bench_module()
    assert set(b.KERNEL_OF) == {"qkv", "out", "up", "down"}
    for name, label in b.KERNEL_OF.items():
        assert b.SYMBOL[label].startswith("k_gemm<")
