"""Register-budget guard of the MFMA and small-batch kernels (no GPU needed):
every instantiation is compiled for gfx950 to assembly and must not reload a
spilled register inside a loop that issues MFMAs (its steady state).  Such a
reload is a vector memory load the compiler waits for with vmcnt(0), which
in the MFMA kernel also waits for every direct-to-LDS copy in flight and
stalls the copy ring, and in the small-batch kernel drains the code loads in
flight once per pair.  Code before and after the loops (set-up, the last
pairs, the epilogue) may reload: it runs once per workgroup."""
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
def _mfma_loops(body):
    """Lines of the kernel's loops that issue MFMAs: the basic blocks of
    every strongly connected component of the control-flow graph that has a
    cycle and contains an MFMA (an out-of-line block that merely jumps back
    is not a loop)."""
    starts = [0]
    for i, l in enumerate(body):
        t = l.strip()
        if re.match(r"^\.LBB\S*:", l) and i not in starts:
            starts.append(i)
        if t.startswith(("s_branch", "s_cbranch", "s_endpgm", "s_setpc")) and i + 1 < len(body):
            starts.append(i + 1)
    starts = sorted(set(starts))
    ends = starts[1:] + [len(body)]
    label = {body[a].split(":")[0]: n for n, a in enumerate(starts) if re.match(r"^\.LBB\S*:", body[a])}
    succ = []
    for n, (a, b) in enumerate(zip(starts, ends)):
        last = next((body[i].strip() for i in range(b - 1, a - 1, -1)
                     if body[i].strip() and not body[i].strip().startswith(";")), "")
        out = []
        m = re.match(r"^s_(cbranch_\w+|branch)\s+(\.LBB\S*)", last)
        if m and m.group(2) in label:
            out.append(label[m.group(2)])
        if not last.startswith(("s_branch", "s_endpgm", "s_setpc")) and n + 1 < len(starts):
            out.append(n + 1)
        succ.append(out)
    # Tarjan's strongly connected components (iterative)
    index, low, on, stack, comps, counter = {}, {}, set(), [], [], [0]
    for root in range(len(starts)):
        if root in index:
            continue
        work = [(root, 0)]
        while work:
            v, k = work.pop()
            if k == 0:
                index[v] = low[v] = counter[0]
                counter[0] += 1
                stack.append(v)
                on.add(v)
            if k < len(succ[v]):
                work.append((v, k + 1))
                w = succ[v][k]
                if w not in index:
                    work.append((w, 0))
                elif w in on:
                    low[v] = min(low[v], index[w])
                continue
            if low[v] == index[v]:
                comp = []
                while True:
                    w = stack.pop()
                    on.discard(w)
                    comp.append(w)
                    if w == v:
                        break
                comps.append(comp)
            if work:
                u = work[-1][0]
                low[u] = min(low[u], low[v])
    lines = []
    for comp in comps:
        if len(comp) == 1 and comp[0] not in succ[comp[0]]:
            continue
        blk = [i for n in comp for i in range(starts[n], ends[n])]
        if any("v_mfma" in body[i] for i in blk):
            lines.extend(blk)
    return sorted(lines)


@pytest.mark.skipif(not shutil.which(HIPCC) and not os.path.exists(HIPCC), reason="no hipcc")
@pytest.mark.parametrize("src", ["ql_gemm.hip", "ql_gemv.hip"])
def test_no_spill_reloads_inside_the_mfma_loop(src, tmp_path):
    bad = []
    n = 0
    for name, body in _kernels(os.path.join(CSRC, src), tmp_path):
        loops = _mfma_loops(body)
        if not loops:
            continue
        n += 1
        inside = [i for i in loops if "scratch_load" in body[i]]
        if inside:
            bad.append((name, len(inside)))
    assert n > 0
    assert not bad, bad
