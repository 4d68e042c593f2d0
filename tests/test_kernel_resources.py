"""Compile-time guard (CPU, no GPU): every HIP kernel in the library keeps its
working set in registers -- no scratch (private memory) spills -- and its
static LDS fits gfx950's 160 KB.  A spill in a streaming or MFMA inner loop
costs more than any tuning gains, so this is checked on every source change."""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_04031_amd", "csrc")
KERNEL_SOURCES = ["tl_repack.hip", "tl_decode.hip", "tl_decode_fp8.hip", "tl_decode_lds.hip", "tl_lgms.hip", "tl_prefill.hip",
                  "tl_view.hip", "tl_stream.hip", "tl_decode_kn.hip"]


@pytest.mark.parametrize("src", KERNEL_SOURCES)
def test_no_scratch_spills_and_lds_fits(src, tmp_path):
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    cmd = [hipcc, "--offload-arch=gfx950", "-O3", "-std=c++17", "-Xclang", "-target-feature",
           "-Xclang", "-packed-fp32-ops", "-I" + os.path.join(ROOT, "include"), "-c", "-x", "hip",
           os.path.join(CSRC, src), "-o", str(tmp_path / "k.o"), "-Rpass-analysis=kernel-resource-usage"]
    out = subprocess.run(cmd, capture_output=True, text=True)
    assert out.returncode == 0, out.stderr[-2000:]
    kernels = re.findall(r"Function Name: (\S+)", out.stderr)
    scratch = [int(x) for x in re.findall(r"ScratchSize \[bytes/lane\]: (\d+)", out.stderr)]
    lds = [int(x) for x in re.findall(r"LDS Size \[bytes/block\]: (\d+)", out.stderr)]
    assert kernels and len(kernels) == len(scratch) == len(lds)
    for name, sc, l in zip(kernels, scratch, lds):
        assert sc == 0, f"{name} spills {sc} bytes/lane"
        assert l <= 160 * 1024, f"{name} uses {l} bytes of LDS"
