"""Register-budget guard of the MFMA and small-batch kernels (no GPU needed):
every instantiation is compiled for gfx950 to assembly and must not reload a
spilled register between its first and last MFMA.  Such a reload is a
vector memory load the compiler waits for with vmcnt(0), which in the MFMA
kernel also waits for every direct-to-LDS copy in flight and stalls the
copy ring."""
import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_30877_amd", "csrc")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _flags():
    sys.path.insert(0, os.path.join(ROOT, "paper_2608_30877_amd"))
    import build  # the library's own compile flags

    return [f for f in build.FLAGS if f not in ("-Wall", "-Wno-unused-function", "-fPIC")]


def _kernels(src, tmp_path):
    out = tmp_path / (os.path.basename(src) + ".s")
    r = subprocess.run([HIPCC, *_flags(), "--cuda-device-only", "-S", src, "-o", str(out)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = out.read_text().splitlines()
    for n, l in enumerate(lines):
        m = re.match(r"^(_Z\S*k_gem[mv]\S*):", l)
        if m:
            end = next(i for i in range(n, len(lines)) if lines[i].startswith(".Lfunc_end"))
            yield m.group(1), lines[n:end]


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="no hipcc")
@pytest.mark.parametrize("src", ["ql_gemm.hip", "ql_gemv.hip"])
def test_no_spill_reloads_inside_the_mfma_loop(src, tmp_path):
    bad = []
    n = 0
    for name, body in _kernels(os.path.join(CSRC, src), tmp_path):
        mf = [i for i, l in enumerate(body) if "v_mfma" in l]
        if not mf:
            continue
        n += 1
        inside = [i for i, l in enumerate(body) if "scratch_load" in l and mf[0] <= i <= mf[-1]]
        if inside:
            bad.append((name, len(inside)))
    assert n > 0
    assert not bad, bad
