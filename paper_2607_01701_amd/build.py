"""Builds libt2vattn in-tree.

* ``libt2vattn.so``: the gfx950 kernels (hipcc) plus the host code, the product library.
* ``libt2vattn_host.so``: the host-only scheduler/validation code (g++), loaded by CPU
  tests that must not need a GPU.

Run ``python -m paper_2607_01701_amd.build`` (or ``__graft_entry__.build()``).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libt2vattn.so")
HOST_LIB = os.path.join(PKG, "libt2vattn_host.so")

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


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in r.stdout.splitlines() if "packed-fp32-ops" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def build(verbose: bool = True) -> None:
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    objs = []
    for s in HIP_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        objs.append(o)
        jobs.append([HIPCC, *HIP_FLAGS, *SCHED.get(s, []), "-c", os.path.join(CSRC, s), "-o", o])
    for s in HOST_SOURCES:
        o = os.path.join(BUILD, s + ".o")
        objs.append(o)
        jobs.append([CXX, *COMMON, "-c", os.path.join(CSRC, s), "-o", o])
    with cf.ThreadPoolExecutor(max_workers=6) as ex:
        for f in [ex.submit(_run, j, verbose) for j in jobs]:
            f.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    tmp = HOST_LIB + ".tmp"
    _run([CXX, *COMMON, "-shared", *(os.path.join(CSRC, s) for s in HOST_SOURCES), "-o", tmp], verbose)
    os.replace(tmp, HOST_LIB)


if __name__ == "__main__":
    build(verbose="-q" not in sys.argv)
