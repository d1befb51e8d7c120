"""Resource budgets the kernels rely on, checked on the compiled code (CPU only: hipcc
cross-compiles for gfx950).  tp_evict runs the lean quantisation beside each score pass: one
score-pass workgroup (8 waves, two per SIMD) and one lean workgroup (4 waves, one per SIMD)
must fit one CU together, in VGPRs (512 per SIMD lane, allocated in granules of 8) and LDS
(160 KB); otherwise the lean kernel waits for free CUs and the overlap is lost."""
import os
import re
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_03276_amd import build  # noqa: E402


def _resources(src, extra=()):
    """{kernel name: (VGPRs, LDS bytes)} from the compiler's resource-usage remarks."""
    cmd = [build.HIPCC, *build.HIP_FLAGS, *extra, "-x", "hip", "-c", os.path.join(build.CSRC, src), "-o",
           os.devnull, "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:]
    out, name = {}, None
    for line in r.stdout.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            out[name] = [None, None]
        m = re.search(r"remark:\s+VGPRs: (\d+)", line)
        if m and name:
            out[name][0] = int(m.group(1))
        m = re.search(r"LDS Size \[bytes/block\]: (\d+)", line)
        if m and name:
            out[name][1] = int(m.group(1))
    return out


def _alloc(vgprs):
    return (vgprs + 7) // 8 * 8


@pytest.fixture(scope="module")
def kernels():
    if not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    res = _resources("quantize.hip")
    res.update(_resources("guide_scores.hip", build.EXTRA_FLAGS.get("guide_scores.hip", [])))
    return res


@pytest.mark.parametrize("kernel", ["k_guide_stats", "k_guide_attn"])
def test_lean_quantisation_fits_beside_score_passes(kernels, kernel):
    passes = {n: v for n, v in kernels.items() if kernel in n}
    leans = {n: v for n, v in kernels.items() if "k_quantize_lean" in n}
    assert passes and leans
    for pn, (pv, plds) in passes.items():
        for ln, (lv, llds) in leans.items():
            assert 2 * _alloc(pv) + _alloc(lv) <= 512, (pn, pv, ln, lv)
            assert plds + llds <= 160 * 1024, (pn, plds, ln, llds)
