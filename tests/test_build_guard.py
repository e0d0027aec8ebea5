"""The build refuses kernels that spill vector registers or use scratch memory (CPU: hipcc
cross-compiles for gfx950 here). The attention kernels order their LDS DMA with counted
vector-memory waits, which spill traffic would silently shift; the guard keeps a future
change from introducing it unnoticed."""
import os
import shutil
import subprocess

import pytest

from paper_2607_01701_amd import build as B

pytestmark = pytest.mark.skipif(not os.path.exists(B.HIPCC) and shutil.which("hipcc") is None,
                                reason="hipcc not available")

# 1024 threads per workgroup leave each wave 128 VGPRs; 160 live accumulators must spill.
SPILLING = r"""
#include <hip/hip_runtime.h>
__global__ __launch_bounds__(1024) void spills(const float* __restrict__ x, float* __restrict__ y, int n) {
  float acc[160];
#pragma unroll
  for (int i = 0; i < 160; ++i) acc[i] = x[threadIdx.x + i * 1024];
  for (int r = 0; r < n; ++r) {
#pragma unroll
    for (int i = 0; i < 160; ++i) acc[i] = acc[i] * acc[(i + 1) % 160] + x[r];
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 160; ++i) s += acc[i] * (i + 1);
  y[threadIdx.x] = s;
}
"""

CLEAN = r"""
#include <hip/hip_runtime.h>
__global__ void clean(const float* __restrict__ x, float* __restrict__ y) { y[threadIdx.x] = 2.0f * x[threadIdx.x]; }
"""


def _compile(tmp_path, name, src):
    p = tmp_path / f"{name}.hip"
    p.write_text(src)
    cmd = [B.HIPCC, *B.HIP_FLAGS, *B.RESOURCE_REMARKS, "-c", str(p), "-o", str(tmp_path / f"{name}.o")]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:]
    return cmd, r.stdout


def test_spilling_kernel_is_rejected(tmp_path):
    cmd, out = _compile(tmp_path, "spills", SPILLING)
    res = B.kernel_resources(out)
    assert any("spills" in k for k in res), out[-2000:]
    bad = B.resource_violations(res)
    assert bad and "spills" in bad[0] and ("Spill" in bad[0] or "Scratch" in bad[0]), bad
    with pytest.raises(RuntimeError, match="spill registers or use scratch"):
        B._run(cmd, verbose=False, check_resources=True)


def test_clean_kernel_passes(tmp_path):
    cmd, out = _compile(tmp_path, "clean", CLEAN)
    res = B.kernel_resources(out)
    assert any("clean" in k for k in res) and not B.resource_violations(res)
    B._run(cmd, verbose=False, check_resources=True)


def test_attention_kernels_are_spill_free(tmp_path):
    """Every kernel of the four attention sources reports no spills and no scratch (the same
    check the build applies)."""
    names = {}
    for src in ("t2v_fwd.hip", "t2v_bwd_pre.hip", "t2v_bwd_dkdv.hip", "t2v_bwd_dq.hip"):
        cmd = [B.HIPCC, *B.HIP_FLAGS, *B.SCHED.get(src, []), *B.RESOURCE_REMARKS, "-c", os.path.join(B.CSRC, src),
               "-o", str(tmp_path / (src + ".o"))]
        r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
        assert r.returncode == 0, r.stdout[-2000:]
        res = B.kernel_resources(r.stdout)
        assert not B.resource_violations(res), B.resource_violations(res)
        names.update(res)
    for kern in ("attn_fwd_kernel", "attn_bwd_pre_kernel", "attn_bwd_dkdv_kernel", "attn_bwd_dq_kernel"):
        assert any(kern in n for n in names), kern
