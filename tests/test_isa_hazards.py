"""Regression test (CPU): no LDS read of the GEMM may have its destination
registers touched while it is in flight.  An LDS-direct variant once reused
such registers right after its main loop, and a late LDS return overwrote an
epilogue address register (a GPU memory fault)."""
import os
import subprocess

import pytest

from conftest import ROOT
from isa_check import hazards, kernel_bodies

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_gemm_asm_reads_are_never_clobbered(tmp_path):
    src = os.path.join(ROOT, "paper_2607_14557_amd", "csrc", "gemm_bf16.hip")
    out = tmp_path / "gemm.s"
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include"), src, "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    kernels = {k: v for k, v in kernel_bodies(out.read_text()).items() if "gemm_bf16_kernel" in k}
    assert len(kernels) >= 6
    for name, body in kernels.items():
        assert sum("ds_read_b128" in l for l in body) > 0, name
        bad = hazards(body)
        assert not bad, "%s: %s" % (name, bad[:3])
