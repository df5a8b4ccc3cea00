"""The library's kernels compiled to gfx950 assembly: no read of a matrix
product's result comes sooner after the product than the compiler's own
spacing, on any path through a branch (tests/isa_hazards.py).  Runs hipcc
without a GPU."""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from isa_hazards import scan
from paper_2510_16292_amd import build as pkg_build

BAD = """\
_Z6kernelv:
\tv_mfma_f32_16x16x32_f16 v[18:21], v[18:21], v[62:65], 0
\ts_cbranch_vccnz .LBB0_2
\tv_mfma_f32_16x16x32_f16 v[2:5], v[2:5], v[62:65], 0
\ts_waitcnt vmcnt(0)
\ts_nop 6
\tv_fmac_f32_e32 v164, v2, v235
.LBB0_2:
\ts_waitcnt vmcnt(0)
\tv_fmac_f32_e32 v171, v18, v235
\ts_endpgm
"""


def test_scanner_flags_the_unpadded_branch_path():
    found = scan(BAD)
    assert [(f[1], f[2], f[3]) for f in found] == [(2, 10, 2)], found
    # padded on the branch path too: nothing to report
    ok = BAD.replace(".LBB0_2:\n", ".LBB0_2:\n\ts_nop 7\n")
    assert scan(ok) == []
    # a read of the second product right after it, in the same block
    near = BAD.replace("\ts_nop 6\n", "")
    assert [(f[1], f[2]) for f in scan(near)] == [(2, 9), (4, 6)]


def _assemble(src, out_dir):
    flags = [f for f in pkg_build.FLAGS if f not in ("-fPIC", "-shared")]
    out = os.path.join(out_dir, os.path.basename(src) + ".s")
    cmd = [pkg_build.hipcc(), *flags, "--cuda-device-only", "-S", "-I", pkg_build.INCLUDE, "-I", pkg_build.CSRC,
           "-o", out, src]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    return out


def test_library_kernels_have_no_short_product_reads(tmp_path):
    try:
        pkg_build.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    srcs = [os.path.join(pkg_build.CSRC, s) for s in pkg_build.SOURCES]
    with ThreadPoolExecutor(max_workers=4) as ex:
        outs = list(ex.map(lambda s: _assemble(s, str(tmp_path)), srcs))
    findings = []
    for o in outs:
        findings += [(os.path.basename(o),) + f for f in scan(open(o).read())]
    assert not findings, findings[:10]
