"""Builds libt2vattn in-tree.

* ``libt2vattn.so``: the gfx950 kernels (hipcc) plus the host code, the product library.
* ``libt2vattn_host.so``: the host-only scheduler/validation code (g++), loaded by CPU
  tests that must not need a GPU.
* ``libt2vattn_checked.so``: the same sources built with ``T2V_CHECKED=1``, a debugging
  variant whose calls validate every work list on the host, check every row the kernels copy
  into LDS on the device, and wait for their kernels (T2V_ERR_BOUNDS on a violation).

Run ``python -m paper_2607_01701_amd.build`` (or ``__graft_entry__.build()``).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libt2vattn.so")
HOST_LIB = os.path.join(PKG, "libt2vattn_host.so")
CHECKED_LIB = os.path.join(PKG, "libt2vattn_checked.so")
CHECKED_FLAGS = ["-DT2V_CHECKED=1"]

HIP_SOURCES = ["t2v_fwd.hip", "t2v_bwd_pre.hip", "t2v_bwd_dkdv.hip", "t2v_bwd_dq.hip", "t2v_api.hip",
               "t2v_probe.hip"]
HOST_SOURCES = ["t2v_host.cpp", "t2v_plan.cpp"]

ARCH = os.environ.get("T2V_OFFLOAD_ARCH", "gfx950")
HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")
CXX = os.environ.get("CXX_HOST", shutil.which("g++") or "g++")

COMMON = ["-O3", "-std=c++17", "-fPIC", "-I", os.path.join(ROOT, "include"), "-Wall"]
# Packed fp32 VALU forms are kept out of generated code. MFMA results stay in ordinary
# VGPRs (the softmax reads them with VALU ops), which avoids AGPR <-> VGPR copies.
HIP_FLAGS = COMMON + [f"--offload-arch={ARCH}", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                      "-mllvm", "-amdgpu-mfma-vgpr-form"]
# Machine-scheduler strategy per kernel, chosen by measurement on MI355X: the ILP-driven
# schedulers interleave LDS reads, MFMAs and softmax arithmetic better, but raise register
# pressure, which only the one-workgroup-per-CU dK/dV kernel can afford in full.
SCHED = {
    "t2v_fwd.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
    "t2v_bwd_dkdv.hip": ["-mllvm", "-amdgpu-sched-strategy=iterative-ilp"],
    "t2v_bwd_dq.hip": ["-mllvm", "-amdgpu-sched-strategy=max-ilp"],
}


# Every kernel is compiled with the compiler's per-kernel resource report, and the build
# fails if any kernel spills vector registers or uses scratch (private) memory. The kernels order
# their LDS DMA with counted `s_waitcnt vmcnt(N)` waits that count only the DMA instructions;
# spill stores and reloads are vector memory operations too. Operations complete in issue
# order, so extra ones only make such a wait stricter (slower), never early; but the kernels'
# register and LDS budgets, their wait depths and their measured speed all assume none, so a
# change that starts spilling is stopped here, on the CPU, before it reaches a GPU.
RESOURCE_REMARKS = ["-Rpass-analysis=kernel-resource-usage"]
_REMARK = re.compile(r"remark:\s+(Function Name|ScratchSize \[bytes/lane\]|SGPRs Spill|VGPRs Spill|"
                     r"Dynamic Stack|VGPRs|AGPRs):\s+(\S+)")


def kernel_resources(compiler_output: str) -> dict:
    """{kernel: {field: value}} from the compiler's kernel-resource-usage remarks."""
    res, cur = {}, None
    for line in compiler_output.splitlines():
        m = _REMARK.search(line)
        if not m:
            continue
        key, val = m.group(1), m.group(2)
        if key == "Function Name":
            cur = res.setdefault(val, {})
        elif cur is not None:
            cur[key] = val
    return res


def resource_violations(resources: dict) -> list:
    """Kernels that spill vector registers or use scratch memory (each as a readable line).
    SGPR spills that stay in VGPR lanes (v_writelane / v_readlane, no scratch) issue no memory
    operations and are allowed; once they reach scratch, ScratchSize is nonzero."""
    bad = []
    for name, r in sorted(resources.items()):
        why = [f"{k} = {r[k]}" for k in ("ScratchSize [bytes/lane]", "VGPRs Spill") if r.get(k, "0") != "0"]
        if r.get("Dynamic Stack", "False") != "False":
            why.append("dynamic stack")
        if why:
            bad.append(f"{name}: {', '.join(why)}")
    return bad


def _run(cmd, verbose, check_resources=False):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    lines = [line for line in r.stdout.splitlines() if "packed-fp32-ops" not in line]
    out = "\n".join(line for line in lines if "kernel-resource-usage" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if check_resources:
        res = kernel_resources(r.stdout)
        bad = resource_violations(res)
        if bad:
            raise RuntimeError("kernels spill registers or use scratch memory (not allowed: the kernels' "
                               "counted LDS-DMA waits and register budgets assume none):\n  " + "\n  ".join(bad))
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose: bool = True) -> None:
    checked_dir = os.path.join(BUILD, "checked")
    os.makedirs(checked_dir, exist_ok=True)
    jobs = []
    objs, checked_objs, host_objs = [], [], []
    for s in HIP_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        objs.append(o)
        jobs.append(([HIPCC, *HIP_FLAGS, *SCHED.get(s, []), *RESOURCE_REMARKS, "-c", os.path.join(CSRC, s), "-o", o],
                     True))
        o = os.path.join(checked_dir, s + ".o")
        checked_objs.append(o)
        jobs.append(([HIPCC, *HIP_FLAGS, *CHECKED_FLAGS, *SCHED.get(s, []), *RESOURCE_REMARKS, "-c",
                      os.path.join(CSRC, s), "-o", o], True))
    for s in HOST_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        host_objs.append(o)
        jobs.append(([CXX, *COMMON, "-c", os.path.join(CSRC, s), "-o", o], False))
    with cf.ThreadPoolExecutor(max_workers=6) as ex:
        for f in [ex.submit(_run, j, verbose, chk) for j, chk in jobs]:
            f.result()
    for lib, hip_objs in ((LIB, objs), (CHECKED_LIB, checked_objs)):
        tmp = lib + ".tmp"
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *hip_objs, *host_objs, "-o", tmp], verbose)
        os.replace(tmp, lib)
    tmp = HOST_LIB + ".tmp"
    _run([CXX, *COMMON, "-shared", *(os.path.join(CSRC, s) for s in HOST_SOURCES), "-o", tmp], verbose)
    os.replace(tmp, HOST_LIB)


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
