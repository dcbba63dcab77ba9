"""Regression test (CPU): no LDS read of the GEMM or the attention kernel may
have its destination registers touched while it is in flight.  An LDS-direct
GEMM variant once reused such registers right after its main loop, and a late
LDS return overwrote an epilogue address register (a GPU memory fault).  The
attention kernel fills its K/V tiles with direct-to-LDS loads and reads V with
LDS transpose reads inside fenced scheduling regions, so it is held to the
same check."""
import os
import subprocess

import pytest

from conftest import ROOT
from isa_check import hazards, kernel_bodies

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _asm(tmp_path, name):
    src = os.path.join(ROOT, "paper_2607_14557_amd", "csrc", name)
    out = tmp_path / (name + ".s")
    from paper_2607_14557_amd.build import FILE_FLAGS
    cmd = [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "--cuda-device-only", "-S",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I" + os.path.join(ROOT, "include")] + FILE_FLAGS.get(name, []) + [src, "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True)
    return kernel_bodies(out.read_text())


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
@pytest.mark.parametrize("src,kernel,min_count,read_op", [
    ("gemm_bf16.hip", "gemm_bf16_kernel", 6, "ds_read_b128"),
    ("gemm_bf16.hip", "gemm_bf16_split_kernel", 4, "ds_read_b128"),
    ("attn_bf16.hip", "attn_bf16_kernel", 1, "ds_read_b64_tr_b16"),
])
def test_lds_reads_are_never_clobbered(tmp_path, src, kernel, min_count, read_op):
    kernels = {k: v for k, v in _asm(tmp_path, src).items() if kernel in k}
    assert len(kernels) >= min_count
    for name, body in kernels.items():
        assert sum(read_op in l for l in body) > 0, name
        bad = hazards(body)
        assert not bad, "%s: %s" % (name, bad[:3])


def test_checker_flags_a_register_reused_in_flight():
    """The checker itself: a read whose destination is overwritten (or read)
    before the lgkmcnt wait that retires it is flagged, across a loop back
    edge too; the same code with the wait in place is clean."""
    clean = """_Zk:
\tds_read_b128 v[4:7], v1
\tds_read_b128 v[8:11], v1 offset:16
\ts_waitcnt lgkmcnt(1)
\tv_add_f32 v12, v4, v5
.LBB0_1:
\ts_waitcnt lgkmcnt(0)
\tv_add_f32 v13, v8, v9
\tds_read_b128 v[8:11], v1 offset:32
\ts_cbranch_scc1 .LBB0_1
\ts_waitcnt lgkmcnt(0)
\tv_mov_b32 v8, 0
\ts_endpgm
.Lfunc_end0:
"""
    assert hazards(kernel_bodies(clean)["_Zk"]) == []
    early = clean.replace("\ts_waitcnt lgkmcnt(1)\n", "")
    assert any("v4" in t for _, _, t in hazards(kernel_bodies(early)["_Zk"]))
    # the back edge brings the loop's last read to the loop head: without the
    # wait there, its first instruction reads v8 in flight
    loop = clean.replace(".LBB0_1:\n\ts_waitcnt lgkmcnt(0)\n", ".LBB0_1:\n")
    assert any("v8" in t for _, _, t in hazards(kernel_bodies(loop)["_Zk"]))
