"""Register budget of the latency-bound kernels (CPU; compiles for gfx950).

The one-launch block kernel, the fused MRConv and the in-register kNN run at
three waves per SIMD, the lean MRConv and the resident-key kNN at four or more, the wide kNN at two; if the register allocator has to spill to scratch
memory to meet that, they slow down without failing any parity test.  This
test compiles their sources with the resource-usage remarks and requires no
scratch for every instantiation of them."""
import os
import re
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2604_21290_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
KERNELS = {"block.hip": "block_kernel", "mrconv.hip": r"13mrconv_kernel|18mrconv_lean_kernel",
           "knn.hip": "knn_kernel", "knn_wide.hip": "knn_wide_kernel",
           "knn_resident.hip": "knn_resident_kernel"}


def _usage(src: str, tmp) -> list:
    out = os.path.join(str(tmp), src + ".o")
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-c",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-Rpass-analysis=kernel-resource-usage", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stderr[-2000:]
    rows, name = [], None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name:
            rows.append((name, int(m.group(1))))
    return rows


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_latency_bound_kernels_do_not_spill(tmp_path):
    with ThreadPoolExecutor(len(KERNELS)) as ex:
        res = dict(zip(KERNELS, ex.map(lambda s: _usage(s, tmp_path), KERNELS)))
    for src, pat in KERNELS.items():
        ks = [(n, sc) for n, sc in res[src] if re.search(pat, n)]
        assert ks, f"no {pat} instantiation found in {src}"
        bad = [(n, sc) for n, sc in ks if sc]
        assert not bad, f"{src}: kernels using scratch: {bad[:4]}"
