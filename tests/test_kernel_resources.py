"""Register budget of the bf16 kernels, from the compiler's resource report (CPU;
the device code is compiled for gfx950 without a GPU).

The GEMM main loop pins the order of its MFMAs, LDS reads and global -> LDS
loads with scheduling fences.  A variant of it once made the compiler rename
the accumulators between two code paths and spill them to scratch memory,
which made the kernel six times slower while every numerical test still
passed.  These checks catch that class of regression: no bf16 MFMA kernel
may use scratch memory, and the tiles that run two waves per SIMD (eight-wave
GEMM tiles, the attention kernels) must still fit two waves per SIMD."""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2206_04959_amd", "csrc")


def _resources(src: str, extra=()):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("needs hipcc")
    cmd = [hipcc, "-std=c++17", "-O3", "--offload-arch=gfx950", "--offload-device-only", "-c",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *extra,
           "-I", CSRC, "-I", os.path.join(ROOT, "include"), os.path.join(CSRC, src), "-o", os.devnull,
           "-Rpass-analysis=kernel-resource-usage"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stderr[-4000:]
    rows, cur = {}, None
    for line in r.stderr.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            cur = m.group(1)
            rows[cur] = {}
            continue
        m = re.search(r"remark:\s+(VGPRs|AGPRs|ScratchSize \[bytes/lane\]|Occupancy \[waves/SIMD\]): (\d+)", line)
        if m and cur:
            rows[cur][m.group(1).split()[0]] = int(m.group(2))
    assert rows, "no resource report"
    return rows


def test_gemm_kernels_do_not_spill():
    rows = _resources("gemm.hip")
    mfma = {k: v for k, v in rows.items() if "gemm_mfma_kernel" in k}
    assert len(mfma) >= 10 * 4 * 6  # every tile x layout x epilogue
    spills = {k: v["ScratchSize"] for k, v in mfma.items() if v.get("ScratchSize", 0) != 0}
    assert not spills, spills
    # the eight-wave tiles the stage uses run two waves per SIMD
    for shape in ("ILi256ELi256ELi2ELi4ELi2E", "ILi256ELi192ELi4ELi2ELi2E", "ILi256ELi128ELi4ELi2ELi3E"):
        occ = {k: v["Occupancy"] for k, v in mfma.items() if shape in k}
        assert occ and min(occ.values()) >= 2, occ


def test_attention_kernels_do_not_spill():
    rows = _resources("attention.hip", extra=("-mllvm", "-amdgpu-mfma-vgpr-form"))
    bf16 = {k: v for k, v in rows.items() if "attn_" in k and "bf16" in k}
    assert len(bf16) == 9  # forward, dQ, dK/dV at d = 64, 96, 128
    spills = {k: v["ScratchSize"] for k, v in bf16.items() if v.get("ScratchSize", 0) != 0}
    assert not spills, spills
    occ = {k: v["Occupancy"] for k, v in bf16.items() if "ILi96E" in k}
    assert occ and min(occ.values()) >= 2, occ
