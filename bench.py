#!/usr/bin/env python3
"""Benchmark of the hot path on one MI355X: packed varlen attention forward + backward.

A step is one t2v_attn_fwd plus one t2v_attn_bwd over the whole packed batch, with all
inputs resident in HBM. The default workload is the heterogeneous mix (16 clips drawn
from three latent grids, 24 heads x 128). Prints one JSON line.

    python bench.py [--steps 50] [--warmup 10] [--workload hetero]

The FLOP count is the usual one for attention with recomputation in the backward:
fwd = 4 H D sum(L^2), bwd = 10 H D sum(L^2), step = 14 H D sum(L^2).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "varlen attention fwd+bwd TFLOP/s and % of bf16 MFMA peak, 1×MI355X"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
# What decides the attention kernels' code and launches: device sources with their launch
# functions, the tile scheduler, and the HIP compile flags (argument validation, the work-list
# cache, the planner and other host-only code are left out).
KERNEL_SOURCES = ("paper_2607_01701_amd/csrc/t2v_fwd.hip", "paper_2607_01701_amd/csrc/t2v_bwd_pre.hip",
                  "paper_2607_01701_amd/csrc/t2v_bwd_dkdv.hip", "paper_2607_01701_amd/csrc/t2v_bwd_dq.hip",
                  "paper_2607_01701_amd/csrc/t2v_kernel_common.hpp", "paper_2607_01701_amd/csrc/t2v_device.hpp",
                  "paper_2607_01701_amd/csrc/t2v_kernels.h",
                  "paper_2607_01701_amd/csrc/t2v_host.cpp", "paper_2607_01701_amd/csrc/t2v_host.h")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def kernel_source_hash() -> str:
    """Hash of the kernel sources and HIP build flags; C++ comments and blank lines are left
    out, so comment edits keep profiles taken on the same code valid."""
    import re

    from paper_2607_01701_amd import build as _build
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        text = "\n".join(line.rstrip() for line in text.splitlines() if line.strip())
        h.update(text.encode())
    flags = [f.replace(_build.ROOT, "<root>") for f in _build.HIP_FLAGS]
    h.update(json.dumps([flags, _build.SCHED], sort_keys=True).encode())
    return h.hexdigest()[:16]


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="hetero", help="tiny | uniform | hetero | long | skew")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="headline workload only: skip the per-workload summary and the fresh-pack comparison")
    ap.add_argument("--write-summaries", nargs="+", metavar=("BENCH_JSON", "SWEEP_JSONL"),
                    help="write the text summaries under profiles/ from a bench line, profiles/hbm_traffic.json "
                         "and (optionally) a --sweep output")
    ap.add_argument("--sweep", action="store_true",
                    help="time every workload (and the natural-order scheduler ablation on the mixed ones); "
                         "one JSON line per run, no CPU baseline")
    ap.add_argument("--cost-model", action="store_true",
                    help="sweep uniform buckets (B clips of S tokens) for three model shapes, fit the attention term "
                         "of the DiT latency model (alpha_2 B S^2 + alpha_1 B S + c0, k = 1) and check it on held-out "
                         "mixed packs; prints a text report")
    ap.add_argument("--plan", action="store_true",
                    help="(CPU) plan one training batch of the heterogeneous mix as a cascade DAG on N GPUs with the "
                         "native genetic-algorithm planner; attention latency from the fitted cost model; compares "
                         "against static parallel degrees and prints a text report")
    ap.add_argument("--balance", action="store_true",
                    help="trace one fwd+bwd step per scheduler order and print each kernel's per-CU busy-time "
                         "CV and idle share (the library's workgroup trace)")
    ap.add_argument("--shares", action="store_true",
                    help="time fwd+bwd at one GPU's share of the long, skew and hetero workloads under k-way head "
                         "sharding (H / k heads, k = 1, 2, 4, 8), with the library's tile choice and forced tiles")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain device copy of known size (for HBM counter scaling)")
    ap.add_argument("--ingest-rocpd", nargs=5, metavar=("KT_DB", "FETCH_DB", "WRITE_DB", "COPY_FETCH_DB",
                                                        "COPY_WRITE_DB"),
                    help="summarise rocprofv3 databases (kernel trace, FETCH_SIZE and WRITE_SIZE of this bench and "
                         "of --copy-calibration) into profiles/; runs on the CPU")
    ap.add_argument("--ingest-mfma", metavar="PMC_DB",
                    help="summarise a rocprofv3 MfmaUtil / MfmaFlopsBF16 counter pass into profiles/; runs on the CPU")
    ap.add_argument("--ingest-sq", nargs=3, metavar=("SQ_A_DB", "SQ_B_DB", "SQ_C_DB"),
                    help="summarise three rocprofv3 SQ counter passes (wave-cycle breakdown, MFMA/VALU co-issue, LDS) "
                         "into profiles/; runs on the CPU")
    return ap.parse_args()


# The paper's own numbers are end-to-end training iteration times on another machine; quoted
# as context only (they measure no attention kernel and are not comparable to this metric).
PAPER_CONTEXT = {
    "hardware": "NVIDIA H100-80GB, 8 GPUs per node (NVLink), 8 x 400 Gbps InfiniBand; PyTorch 2.7.1, CUDA 12.6; "
                "16 GPUs end to end, up to 64 for scalability",
    "avg_iteration_time_s": {"HunyuanVideo-13B stage 1 (360p)": 22.07, "stage 2 (720p)": 32.96,
                             "stage 3 (1080p)": 26.80},
    "iteration_time_reduction_vs": {"Megatron-LM": "up to 65%", "DeepSpeed": "up to 59%", "FlexSP": "up to 35%"},
    "case_study_step_s": {"static DP=4 x SP=4 slowest rank": 58.6, "fastest rank": 6.0, "FlexSP": 45.2,
                          "Arachne": 31.4},
    "note": "Section V-B (end-to-end), V-D (ablation table) and V-E / Section III (case study: static, FlexSP "
            "and Arachne schedules of one step); no attention-kernel time or throughput is published, so "
            "vs_baseline is null",
}


def kernel_flops(H, D, ssq):
    """Algorithmic work per launch of each kernel (MFMA flops, or bytes for Delta)."""
    base = H * D * ssq
    return {"fwd": 4 * base, "bwd_dkdv": 8 * base, "bwd_dq": 6 * base}


def cpu_baseline(pack, budget_s: float = 15.0):
    """The float64 oracle, untuned, on a bounded sample of the same workload's (clip, head) pairs.

    The shortest clip calibrates the oracle's rate; then clips are taken longest first,
    skipping any whose predicted time exceeds the remaining budget, cycling over heads.
    Clips longer than 32,768 tokens are cut to their first 8,192 tokens (a shorter clip of
    the same statistics), so the sample stays bounded.
    """
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:  # pragma: no cover
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    cu = pack.cu_seqlens
    cuk = cu if pack.cu_seqlens_k is None else pack.cu_seqlens_k
    lens = np.diff(cu).astype(np.int64)
    lens_k = np.diff(cuk).astype(np.int64)
    q, k, v, g = (pack.f32(n) for n in ("q", "k", "v", "dout"))
    done, flops, t_used = [], 0.0, 0.0

    def keys_of(s, n):  # self-attention: the (possibly cut) clip itself; cross: the sequence's keys
        return n if pack.cu_seqlens_k is None else int(lens_k[s])

    def run(s, h):
        nonlocal flops, t_used
        a, ka = int(cu[s]), int(cuk[s])
        n = int(min(lens[s], 8192 if lens[s] > 32768 else lens[s]))
        nk = keys_of(s, n)
        t0 = time.perf_counter()
        oracle.head_forward_backward(q[a:a + n, h], k[ka:ka + nk, h], v[ka:ka + nk, h], g[a:a + n, h], pack.scale)
        dt = time.perf_counter() - t0
        t_used += dt
        fl = 14.0 * pack.head_dim * float(n) * float(nk)
        flops += fl
        done.append((n, h))
        return dt, fl

    nz = [int(s) for s in np.argsort(lens, kind="stable") if lens[s] > 0]
    dt, f0 = run(nz[0], 0)
    rate = f0 / max(dt, 1e-9)
    distinct = []
    for s in sorted(nz, key=lambda s: -lens[s]):
        if int(lens[s]) not in [int(lens[x]) for x in distinct]:
            distinct.append(s)
    h = 0
    progress = True
    while t_used < budget_s and progress:
        progress = False
        h = (h + 1) % pack.heads
        for s in distinct:
            n = min(lens[s], 8192 if lens[s] > 32768 else lens[s])
            if 14.0 * pack.head_dim * float(n) * float(keys_of(s, int(n))) / rate <= budget_s - t_used:
                dt, fl = run(s, h)
                rate = fl / max(dt, 1e-9)
                progress = True
            if t_used >= budget_s:
                break
    return {"value": flops / t_used * 1e-12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "seconds": round(t_used, 3),
            "gflops_strict_no_recompute": round(flops * 12.0 / 14.0 / t_used * 1e-9, 2),
            "host": host_info(),
            "sample": f"{len(done)} (clip query tokens, head) pairs of this workload {done}; float64 numpy oracle "
                      f"fwd+bwd, counted at the same 14*D*Lq*Lk per pair"}


def host_info() -> dict:
    """CPU model, logical CPU count and BLAS library of the host the oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        from threadpoolctl import threadpool_info
        b = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if b:
            blas = f"{b[0].get('internal_api')} {b[0].get('version')} ({b[0].get('num_threads')} threads)"
    except Exception:  # pragma: no cover
        pass
    return {"cpu_model": model, "nproc": os.cpu_count(), "blas": blas}


def copy_calibration():
    """A plain device-to-device copy of 1 GiB, 5 times, for scaling HBM byte counters."""
    import torch
    n = 1 << 30
    src = torch.ones(n // 2, dtype=torch.bfloat16, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "launches": 5}), flush=True)


SLOT_OF_KERNEL = {"attn_fwd_kernel": "fwd", "attn_bwd_pre_kernel": "bwd_pre", "attn_bwd_dkdv_kernel": "bwd_dkdv",
                  "attn_bwd_dq_kernel": "bwd_dq"}


def _slot(name):
    for key, slot in SLOT_OF_KERNEL.items():
        if key in name:
            return slot
    return None


def ingest_rocpd(kt_db, fetch_db, write_db, copy_fetch_db, copy_write_db, workload):
    """Per-kernel durations and HBM bytes from rocprofv3 (rocpd SQLite) output.

    FETCH_SIZE / WRITE_SIZE are scaled by what they read for a plain copy of known size.
    Writes profiles/hbm_traffic.json (read by the bench) and prints a text summary.
    """
    import sqlite3

    def counters(db):
        c = sqlite3.connect(db)
        rows = c.execute("select kernel_name, counter_name, count(*), avg(value) from counters_collection "
                         "group by kernel_name, counter_name").fetchall()
        c.close()
        return rows

    copy_bytes = 1 << 30
    cf = [r for r in counters(copy_fetch_db) if "copyBuffer" in r[0]]
    cw = [r for r in counters(copy_write_db) if "copyBuffer" in r[0]]
    f_scale = copy_bytes / (cf[0][3] * 1024.0)
    w_scale = copy_bytes / (cw[0][3] * 1024.0)
    kt = sqlite3.connect(kt_db)
    trace = kt.execute("select name, count(*), avg(end-start), min(end-start), max(end-start) from kernels "
                       "group by name").fetchall()
    kt.close()
    kernels = {}
    lines = [f"kernel-trace (ns -> ms)          launches    avg_ms     min_ms     max_ms"]
    for name, n, avg, mn, mx in sorted(trace, key=lambda r: -r[1] * r[2]):
        slot = _slot(name)
        if slot:
            kernels.setdefault(slot, {})["trace_avg_ms"] = avg / 1e6
            lines.append(f"  {slot:28s} {n:8d} {avg / 1e6:10.4f} {mn / 1e6:10.4f} {mx / 1e6:10.4f}")
    for rows, key, scale in ((counters(fetch_db), "fetch", f_scale), (counters(write_db), "write", w_scale)):
        for name, cname, n, avg_kb in rows:
            slot = _slot(name)
            if slot:
                kernels.setdefault(slot, {})[f"{key}_kib_raw"] = avg_kb
                kernels[slot][f"{key}_bytes"] = avg_kb * 1024.0 * scale
    lines.append(f"HBM counters per launch (copy-scaled: FETCH x{f_scale:.4f}, WRITE x{w_scale:.4f})")
    for slot, k in kernels.items():
        if "fetch_bytes" in k and "write_bytes" in k:
            k["hbm_bytes_per_launch"] = k["fetch_bytes"] + k["write_bytes"]
            lines.append(f"  {slot:28s} fetch {k['fetch_bytes'] / 1e9:8.3f} GB  write {k['write_bytes'] / 1e9:8.3f} GB"
                         f"  total {k['hbm_bytes_per_launch'] / 1e9:8.3f} GB")
    rec = {"workload": workload, "kernel_source_hash": kernel_source_hash(), "fetch_scale": f_scale,
           "write_scale": w_scale, "copy_bytes": copy_bytes, "kernels": kernels}
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)
    print("\n".join(lines))


def mfma_cmd(out):
    """The counter pass summarised by --ingest-mfma, writing under directory `out`."""
    return (f"rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 SQ_INSTS_MFMA -d {out}/pmc_mfma -o m -- "
            "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-extras")


def ingest_mfma(pmc_db, workload):
    """MFMA utilisation per kernel from a rocprofv3 counter pass (derived metrics MfmaUtil =
    MFMA-busy cycles / (GPU-active cycles x SIMDs), MfmaFlopsBF16 = bf16 MFMA ops x 512);
    durations from profiles/hbm_traffic.json (same kernel sources). Writes the text summary
    profiles/attn_fwd_<workload>_mfma_counters.txt."""
    import sqlite3

    from paper_2607_01701_amd.workload import DESCRIPTIONS, workload_shape

    _, lengths, H, D = workload_shape(workload)
    ssq = int(sum(int(x) * int(x) for x in lengths))
    kf = kernel_flops(H, D, ssq)
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    if t["kernel_source_hash"] != kernel_source_hash() or t.get("workload") != workload:
        raise SystemExit("profiles/hbm_traffic.json comes from other kernel sources or another workload")
    c = sqlite3.connect(pmc_db)
    rows = c.execute("select kernel_name, counter_name, count(*), avg(value) from counters_collection "
                     "group by kernel_name, counter_name").fetchall()
    c.close()
    by = {}
    for name, cname, n, avg in rows:
        slot = _slot(name)
        if slot:
            by.setdefault(slot, {})[cname] = (avg, n)
    lines = [f"rocprofv3 MFMA counters: attention kernels, {workload} workload ({DESCRIPTIONS[workload]})",
             f"Kernel source hash (bench.py kernel_source_hash): {kernel_source_hash()}", "",
             "Commands (repo root, on the GPU):", "  " + mfma_cmd(os.path.dirname(os.path.dirname(pmc_db)) or "."),
             f"  python3 bench.py --ingest-mfma {pmc_db} --workload {workload}",
             "Durations: kernel-trace averages of the same sources (profiles/hbm_traffic.json).", "",
             f"{'kernel':10s} {'MfmaUtil %':>10s} {'MFMA flops/launch':>18s} {'algorithmic':>12s} {'ratio':>6s} "
             f"{'trace ms':>9s} {'counter TF/s':>12s} {'% of 2.5 PF':>11s}"]
    for slot in ("bwd_dkdv", "bwd_dq", "fwd"):
        d = by.get(slot, {})
        util = d.get("MfmaUtil", (float("nan"), 0))[0]
        fl = d.get("MfmaFlopsBF16", (float("nan"), 0))[0]
        ms = t["kernels"][slot]["trace_avg_ms"]
        tf = fl / (ms * 1e-3) * 1e-12
        lines.append(f"{slot:10s} {util:10.1f} {fl:18.4e} {kf[slot]:12.4e} {fl / kf[slot]:6.3f} {ms:9.3f} "
                     f"{tf:12.0f} {100 * tf / PEAK_BF16_TFLOPS:10.1f}%")
    lines += ["", "MfmaUtil is the share of SIMD cycles with the matrix unit busy at the clock the chip ran; "
              "'% of 2.5 PF' is the counter-measured MFMA rate against the published bf16 dense peak "
              "(which assumes the 2.4 GHz peak clock).",
              "Algorithmic executed MFMA work per launch: fwd 4, dK/dV 8, dQ 6 x H*D*sum(L^2) = "
              f"{H}*{D}*{ssq:,}; ratio = counter flops / algorithmic (1.000 means no MFMA work beyond "
              "the design's products, masked tails included)."]
    out = os.path.join(ROOT, "profiles", f"attn_fwd_bwd_{workload}_mfma_counters.txt")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


SQ_PASSES = (
    "SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY SQ_ACTIVE_INST_VALU "
    "SQ_ACTIVE_INST_LDS SQ_ACTIVE_INST_MISC",
    "SQ_VALU_MFMA_BUSY_CYCLES SQ_VALU_MFMA_COEXEC_CYCLES SQ_WAIT_INST_LDS SQ_LDS_IDX_ACTIVE SQ_LDS_BANK_CONFLICT "
    "SQ_LDS_DATA_FIFO_FULL SQ_LDS_CMD_FIFO_FULL SQ_INST_LEVEL_LDS",
    "SQ_INSTS_VALU SQ_INSTS_LDS SQ_INSTS_MFMA SQ_INSTS_SALU SQ_INSTS_VMEM SQ_THREAD_CYCLES_VALU SQ_ACTIVE_INST_SCA "
    "SQ_ACTIVE_INST_VMEM",
)


def ingest_sq(dbs, workload):
    """Per-kernel SQ counter summary (three passes of at most eight SQ counters each):
    where the waves' cycles go, how often the matrix core and the VALU work at once, and how
    busy the LDS is. Writes profiles/attn_fwd_bwd_<workload>_sq_counters.txt."""
    import sqlite3

    by = {}
    for db in dbs:
        c = sqlite3.connect(db)
        rows = c.execute("select kernel_name, counter_name, count(*), avg(value) from counters_collection "
                         "group by kernel_name, counter_name").fetchall()
        c.close()
        for name, cname, n, avg in rows:
            slot = _slot(name)
            if slot:
                by.setdefault(slot, {})[cname] = avg
    cmds = [f"rocprofv3 --pmc {p} -d <out>/pmc_sq{x} -o {x} -- python3 bench.py --steps 2 --warmup 1 "
            "--no-cpu-baseline --no-extras" for p, x in zip(SQ_PASSES, "abc")]
    lines = [f"rocprofv3 SQ counters: attention kernels, {workload} workload, averages per launch.",
             f"Kernel source hash (bench.py kernel_source_hash): {kernel_source_hash()}", "",
             "Commands (repo root, on the GPU):"] + ["  " + c for c in cmds] + [
             f"  python3 bench.py --ingest-sq <out>/pmc_sqa/a_results.db <out>/pmc_sqb/b_results.db "
             f"<out>/pmc_sqc/c_results.db --workload {workload}", ""]
    order = ("bwd_dkdv", "bwd_dq", "fwd", "bwd_pre")
    names = sorted({k for d in by.values() for k in d})
    lines.append(f"{'counter':30s} " + " ".join(f"{n:>14s}" for n in order))
    for cn in names:
        lines.append(f"{cn:30s} " + " ".join(f"{by.get(n, {}).get(cn, float('nan')):14.4g}" for n in order))
    lines += ["", "Ratios (per kernel):"]

    def ratio(n, a, b):
        d = by.get(n, {})
        return d[a] / d[b] if d.get(b) else float("nan")

    for label, a, b in (("waiting (any) / wave cycles", "SQ_WAIT_ANY", "SQ_WAVE_CYCLES"),
                        ("waiting for issue / wave cycles", "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES"),
                        ("issuing (any) / wave cycles", "SQ_ACTIVE_INST_ANY", "SQ_WAVE_CYCLES"),
                        ("VALU issue / wave cycles", "SQ_ACTIVE_INST_VALU", "SQ_WAVE_CYCLES"),
                        ("LDS issue / wave cycles", "SQ_ACTIVE_INST_LDS", "SQ_WAVE_CYCLES"),
                        ("waiting for LDS issue / wave cycles", "SQ_WAIT_INST_LDS", "SQ_WAVE_CYCLES"),
                        ("MFMA-VALU co-execution / MFMA busy", "SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES"),
                        ("LDS bank conflict / LDS active", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE"),
                        ("LDS active / busy cycles", "SQ_LDS_IDX_ACTIVE", "SQ_BUSY_CYCLES"),
                        ("LDS instructions / MFMA", "SQ_INSTS_LDS", "SQ_INSTS_MFMA"),
                        ("VALU instructions / MFMA", "SQ_INSTS_VALU", "SQ_INSTS_MFMA")):
        lines.append(f"  {label:38s} " + " ".join(f"{ratio(n, a, b):14.3f}" for n in order))
    out = os.path.join(ROOT, "profiles", f"attn_fwd_bwd_{workload}_sq_counters.txt")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def profile_cmds(out):
    """The kernel-trace and HBM-counter passes summarised by --ingest-rocpd and
    --write-summaries, writing under directory `out`."""
    return f"""Commands (repo root, on the GPU; rocprofv3 writes rocpd SQLite files):
  rocprofv3 --kernel-trace --stats -d {out}/prof_kt -o kt -- python3 bench.py --steps 20 --warmup 5 --no-cpu-baseline --no-extras
  rocprofv3 --pmc FETCH_SIZE -d {out}/pmc_fetch -o f -- python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-extras
  rocprofv3 --pmc WRITE_SIZE -d {out}/pmc_write -o w -- python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline --no-extras
  rocprofv3 --pmc FETCH_SIZE -d {out}/pmc_copy_fetch -o cf -- python3 bench.py --copy-calibration
  rocprofv3 --pmc WRITE_SIZE -d {out}/pmc_copy_write -o cw -- python3 bench.py --copy-calibration
  python3 bench.py --steps 20 --warmup 5 > {out}/bench_hetero.json
Summarised with:
  python3 bench.py --ingest-rocpd {out}/prof_kt/kt_results.db {out}/pmc_fetch/f_results.db \\
      {out}/pmc_write/w_results.db {out}/pmc_copy_fetch/cf_results.db {out}/pmc_copy_write/cw_results.db
  python3 bench.py --write-summaries {out}/bench_hetero.json {out}/sweep.jsonl
"""


def write_summaries(bench_json, sweep_jsonl=None):
    """Text summaries under profiles/ from a bench line, profiles/hbm_traffic.json and a sweep."""
    with open(bench_json) as f:
        b = json.loads([x for x in f.read().strip().splitlines() if x.startswith("{")][-1])
    with open(TRAFFIC_FILE) as f:
        t = json.load(f)
    if t["kernel_source_hash"] != b["kernel_source_hash"]:
        raise SystemExit("the counters and the bench line come from different kernel sources")
    k, bk = t["kernels"], b["kernels"]
    c = b["config"]
    H, D, T, ssq = c["heads"], c["head_dim"], c["total_tokens"], c["sum_sq_len"]
    hds = H * D * ssq
    alg = {"fwd": 4 * hds, "bwd_dkdv": 8 * hds, "bwd_dq": 6 * hds}
    head = ("attention forward + backward kernels, heterogeneous mix workload\n"
            "(16 clips: 6x1,280 + 7x6,912 + 3x20,280 tokens, 24 heads x 128, bf16), one MI355X.\n"
            f"Kernel source hash (bench.py kernel_source_hash): {t['kernel_source_hash']}\n\n"
            + profile_cmds(os.path.dirname(bench_json) or ".") + "\n")
    order = ("bwd_dkdv", "bwd_dq", "fwd", "bwd_pre")
    lines = ["rocprofv3 kernel trace: " + head, "kernel-trace averages (ms per launch):"]
    lines += [f"  {n:10s} {k[n]['trace_avg_ms']:10.4f}" for n in order]
    lines.append("bench.py live HIP-event averages (separate run of the same sources, "
                 f"{b['steps']} timed steps):")
    lines.append("  " + "   ".join(f"{n} {bk[n]['avg_ms']:.3f} ms" for n in order))
    lines.append(f"Algorithmic MFMA work per launch (H*D*sum(L^2) = {H}*{D}*{ssq:,}):")
    lines.append("  " + ", ".join(f"{n} {alg[n] / 1e12:.2f} TFLOP" for n in ("fwd", "bwd_dkdv", "bwd_dq")))
    lines.append("  -> " + ", ".join(f"{n} {alg[n] / (k[n]['trace_avg_ms'] * 1e-3) / 1e12:.0f} TFLOP/s"
                                    for n in ("fwd", "bwd_dkdv", "bwd_dq")) + " at the trace averages (peak 2500).")
    lines.append(f"Whole step (bench.py): {b['ms_per_step']:.2f} ms = {b['value']:.0f} TFLOP/s at 14*H*D*sum(L^2).")
    with open(os.path.join(ROOT, "profiles", "attn_fwd_bwd_hetero_kernel_trace.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")

    tb = T * H * D * 2 / 1e6
    lb = T * H * 4 / 1e6
    ab = {"fwd": 4 * tb + lb, "bwd_pre": 2 * tb + 3 * lb, "bwd_dkdv": 6 * tb + 2 * lb, "bwd_dq": 5 * tb + 2 * lb}
    lines = ["rocprofv3 HBM byte counters: " + head,
             f"Copy calibration: a {t['copy_bytes'] >> 20} MiB device-to-device copy scales FETCH_SIZE by "
             f"{t['fetch_scale']:.4f} and WRITE_SIZE by {t['write_scale']:.4f}.", "",
             "HBM bytes per launch (copy-scaled FETCH_SIZE + WRITE_SIZE) against the algorithmic bytes "
             "(each input read once, each output written once):"]
    for n in order:
        lines.append(f"  {n:10s} fetch {k[n]['fetch_bytes'] / 1e9:7.3f} GB  write {k[n]['write_bytes'] / 1e9:7.3f} GB"
                     f"  total {k[n]['hbm_bytes_per_launch'] / 1e9:7.3f} GB   algorithmic {ab[n] / 1e3:6.3f} GB"
                     f"   {k[n]['hbm_bytes_per_launch'] / (k[n]['trace_avg_ms'] * 1e-3) / 1e12:5.2f} TB/s")
    lines += ["Algorithmic: fwd q,k,v,out + lse; bwd_pre out,dout + Delta, lse*log2e (and the lse read);",
              "bwd_dkdv q,k,v,dout,dk,dv + lse2, Delta; bwd_dq q,k,v,dout,dq + lse2, Delta.",
              "The MFMA kernels re-read K/V (fwd, dQ) or Q/dO (dK/dV) once per 128-row tile, mostly from L2 and",
              "the MALL; their HBM rates sit far below the 8 TB/s peak, so they are not bandwidth bound.",
              "The Delta pass is HBM-bound; a workgroup owns one head and 64 consecutive tokens, so its [H, T]",
              "stores and lse reads are contiguous 256-byte runs."]
    with open(os.path.join(ROOT, "profiles", "attn_fwd_bwd_hetero_hbm_counters.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")

    if sweep_jsonl:
        with open(sweep_jsonl) as f:
            rows = [json.loads(x) for x in f if x.startswith("{")]
        out = ["bench.py --sweep: every workload, fwd + bwd, one MI355X, bf16 in / fp32 accumulate, synthetic "
               "N(0,1) inputs.", f"Kernel source hash (bench.py kernel_source_hash): {rows[0]['kernel_source_hash']}",
               "", "Command (repo root, on the GPU):", f"  python3 bench.py --sweep > {sweep_jsonl}",
               f"  python3 bench.py --write-summaries {bench_json} {sweep_jsonl}",
               "(one JSON line per run; warmup = min(10, steps / 2); HIP events on the launch stream)", "",
               "FLOP convention: fwd 4*H*D*sum(L^2), bwd 10*H*D*sum(L^2), step 14*H*D*sum(L^2); % of the "
               "2.5 PFLOP/s bf16 dense peak.", "",
               f"{'workload':9s} {'order':14s} {'steps':>5s} {'ms/step':>10s} {'step TF/s':>10s} {'% peak':>7s} "
               f"{'fwd TF/s':>9s} {'bwd TF/s':>9s}  kernels fwd / dK,dV / dQ (executed-MFMA TF/s), Delta GB/s"]
        vals = {}
        for r in rows:
            cc, kk = r["config"], r["kernels"]
            name = cc["workload"].split(":")[0]
            vals[(name, cc["scheduler_order"])] = r["value"]
            ks = (f"{kk['fwd']['tflops']:.0f} / {kk['bwd_dkdv']['tflops']:.0f} / {kk['bwd_dq']['tflops']:.0f}, "
                  f"{kk['bwd_pre']['gbs']:.0f}")
            out.append(f"{name:9s} {cc['scheduler_order']:14s} {r['steps']:5d} {r['ms_per_step']:10.3f} "
                       f"{r['value']:10.1f} {100 * r['frac_of_peak']:6.1f}% {r['fwd_tflops']:9.1f} "
                       f"{r['bwd_tflops']:9.1f}  {ks}")
        out += ["", "Scheduler ablation (T2V_ORDER=natural vs the default longest-first order):"]
        for name in ("hetero", "skew"):
            a_, n_ = vals.get((name, "longest_first")), vals.get((name, "natural"))
            if a_ and n_:
                out.append(f"  {name:7s} {a_:.1f} vs {n_:.1f} TFLOP/s ({100 * (a_ / n_ - 1):+.1f}% for longest-first)")
        out.append("The tiny pack (640 tokens, 2 heads) is launch-bound: four launches take ~0.08 ms in all.")
        with open(os.path.join(ROOT, "profiles", "attn_all_workloads_sweep.txt"), "w") as f:
            f.write("\n".join(out) + "\n")


# Model shapes of the paper's Table II (hidden size / heads = head_dim): 1536/12, 3072/24, 1920/30.
COST_SHAPES = ((12, 128), (24, 128), (30, 64))
# Table II: model, layers, heads, head_dim (hidden = heads x head_dim).
TABLE2_MODELS = (("Wan2.1-1.3B", 30, 12, 128), ("CogVideoX-5B", 30, 30, 64), ("HunyuanVideo-13B", 60, 24, 128))
GEMM_TOKENS = (4096, 16384, 65536)
DIT_COST_FILE = os.path.join(ROOT, "profiles", "dit_cost_model.json")


def gemm_proxy_sweep(steps: int = 5, warmup: int = 2):
    """alpha_1 of Eq. (9), measured: the linear operations of one DiT block, forward and
    backward, as bf16 GEMMs on the GPU (torch.matmul, i.e. the vendor BLAS; a measurement
    outside libt2vattn). Per token of hidden size d: the QKV projection (d x 3d), the attention
    output projection (d x d) and the MLP (d x 4d, 4d x d), each forward (X W), and backward
    (dX = dY W^T, dW = X^T dY): 72 d^2 flops per token. Fits t_ms = alpha1 * tokens + c per
    Table II hidden size over GEMM_TOKENS tokens. Returns {hidden: (alpha1_ms_per_token, c_ms,
    TFLOP/s at the largest size, rows)}."""
    import numpy as np
    import torch

    out = {}
    for name, layers, H, D in TABLE2_MODELS:
        d = H * D
        gen = torch.Generator(device="cuda").manual_seed(d)
        shapes = [(d, 3 * d), (d, d), (d, 4 * d), (4 * d, d)]
        W = [torch.randn(a, b, generator=gen, device="cuda").to(torch.bfloat16) / a ** 0.5 for a, b in shapes]
        rows = []
        for n in GEMM_TOKENS:
            X = [torch.randn(n, a, generator=gen, device="cuda").to(torch.bfloat16) for a, _ in shapes]
            dY = [torch.randn(n, b, generator=gen, device="cuda").to(torch.bfloat16) for _, b in shapes]
            Wt = [w.t().contiguous() for w in W]
            Xt = [x.t().contiguous() for x in X]  # every operand contiguous (no transposed views)

            def block():
                for x, xt, w, wt, dy in zip(X, Xt, W, Wt, dY):
                    torch.matmul(x, w)            # forward
                    torch.matmul(dy, wt)          # dX
                    torch.matmul(xt, dy)          # dW

            for _ in range(warmup):
                block()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(steps):
                block()
            e1.record()
            torch.cuda.synchronize()
            ms = e0.elapsed_time(e1) / steps
            rows.append((n, ms))
            print(f"[cost-model] GEMM proxy d={d} tokens={n}: {ms:.3f} ms "
                  f"({72.0 * d * d * n / (ms * 1e-3) * 1e-12:.0f} TFLOP/s)", file=sys.stderr, flush=True)
            del X, Xt, dY, Wt
        A = np.array([[n, 1.0] for n, _ in rows])
        t = np.array([ms for _, ms in rows])
        w = 1.0 / t
        coef, *_ = np.linalg.lstsq(A * w[:, None], t * w, rcond=None)
        n_big, ms_big = rows[-1]
        out[d] = (float(coef[0]), float(coef[1]), 72.0 * d * d * n_big / (ms_big * 1e-3) * 1e-12, rows)
        del W
        torch.cuda.empty_cache()
    return out
COST_SEQ = (1024, 2048, 4096, 8192, 16384, 32768)
COST_BATCH = (1, 2, 4, 8)
COST_MAX_TOKENS = 65536


def cost_model_sweep(steps: int = 4, warmup: int = 2):
    """Time fwd+bwd of libt2vattn on uniform buckets and mixed packs; fit and validate the
    attention latency model (paper Section IV-B, Eq. (9), the alpha_2 B S^2 term at k = 1)."""
    import numpy as np
    import torch

    from paper_2607_01701_amd import _lib, costmodel
    from paper_2607_01701_amd.workload import cu_from_lengths, workload_shape

    L = _lib.lib()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    rng = np.random.default_rng(0)
    heldout = []  # mixed packs: the hetero mix at four seeds, skewed mixes, one long clip
    for seed in range(4):
        heldout.append(("hetero seed %d" % seed, workload_shape("hetero", seed)[1]))
    heldout.append(("1 x 75,600 (21x45x80)", [75600]))
    heldout.append(("20,280 + 32 x 1,024", [20280] + [1024] * 32))
    heldout.append(("random 1k-16k x 12", rng.integers(1024, 16385, size=12).tolist()))

    def time_pack(lengths, H, D, bufs):
        cu = np.ascontiguousarray(cu_from_lengths(lengths), dtype=np.int32)
        T, nseq = int(cu[-1]), len(lengths)
        cup = cu.ctypes.data_as(_lib._i32p)
        q, k, v, g, out, dq, dk, dv, lse, ws = bufs
        sc = 1.0 / D ** 0.5

        def step():
            st = L.t2v_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cup, nseq, H, D, sc, out.data_ptr(),
                                lse.data_ptr(), sh)
            if st:
                raise _lib.T2VError(st, _lib.t2v_last_error())
            st = L.t2v_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(), cup, nseq,
                                H, D, sc, g.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), ws.data_ptr(), sh)
            if st:
                raise _lib.T2VError(st, _lib.t2v_last_error())

        for _ in range(warmup):
            step()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            step()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps

    fit_samples, val_samples = [], []
    lines = []
    for H, D in COST_SHAPES:
        tmax = max(COST_MAX_TOKENS, max(sum(l) for _, l in heldout))
        gen = torch.Generator(device="cuda").manual_seed(H * 1000 + D)
        bufs = [torch.randn((tmax, H, D), generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)
                for _ in range(4)]
        bufs += [torch.empty((tmax, H, D), dtype=torch.bfloat16, device="cuda") for _ in range(4)]
        bufs += [torch.empty((H, tmax), dtype=torch.float32, device="cuda"),
                 torch.empty((2, H, tmax), dtype=torch.float32, device="cuda")]
        for S in COST_SEQ:
            for B in COST_BATCH:
                if B * S > COST_MAX_TOKENS:
                    continue
                ms = time_pack([S] * B, H, D, bufs)
                fit_samples.append(([S] * B, H, D, ms))
                print(f"[cost-model] H={H} D={D} B={B} S={S}: {ms:.3f} ms", file=sys.stderr, flush=True)
        for name, lengths in heldout:
            ms = time_pack(lengths, H, D, bufs)
            val_samples.append((lengths, H, D, ms, name))
            print(f"[cost-model] H={H} D={D} {name}: {ms:.3f} ms", file=sys.stderr, flush=True)
        del bufs
        torch.cuda.empty_cache()

    # One fit per model shape: the kernels' efficiency differs between head dims (the paper
    # likewise fits its regression coefficients for the model being trained).
    lines.append("Command (repo root, on the GPU): python3 bench.py --cost-model")
    lines.append(f"Kernel source hash (bench.py kernel_source_hash): {kernel_source_hash()}")
    lines.append("")
    lines.append("Attention term of the DiT latency model (Section IV-B, Eq. (9)) on one MI355X (k = 1),")
    lines.append("fwd + bwd of libt2vattn in bf16, fitted per model shape of Table II:")
    lines.append("  t_ms = alpha2 * sum(L^2) + alpha1 * sum(L) + c0   (a bucket of B clips of S tokens: sum(L^2) = B*S^2)")
    lines.append(f"  fit set: uniform buckets, S in {list(COST_SEQ)}, B in {list(COST_BATCH)}, B*S <= {COST_MAX_TOKENS}; "
                 "rows weighted by 1/t (relative error)")
    lines.append("  held-out set: mixed packs not used in the fit")
    lines.append("")
    all_val = []
    for H, D in COST_SHAPES:
        fs = [x for x in fit_samples if x[1] == H and x[2] == D]
        vs = [x for x in val_samples if x[1] == H and x[2] == D]
        model, stats = costmodel.fit(fs)
        ve = costmodel.relative_errors(model, [x[:4] for x in vs])
        all_val.extend(ve.tolist())
        lines.append(f"H={H} D={D}: alpha2 = {model.alpha2(H, D):.6e} ms/token^2  alpha1 = {model.alpha1(H, D):.6e} "
                     f"ms/token  c0 = {model.c0:.4f} ms")
        lines.append(f"  large-S throughput 14*H*D/alpha2 = {14.0 * H * D / (model.alpha2(H, D) * 1e-3) * 1e-12:.0f} "
                     f"TFLOP/s; fit rms {100 * stats['rms_rel_err']:.2f}% max {100 * stats['max_rel_err']:.2f}%; "
                     f"held-out rms {100 * float(np.sqrt(np.mean(ve ** 2))):.2f}% max {100 * float(np.max(np.abs(ve))):.2f}%")
        lines.append("    B      S   measured_ms  predicted_ms  rel_err")
        for (l, _, _, ms) in fs:
            pr = model.predict_lengths(l, H, D)
            lines.append(f"  {len(l):3d} {l[0]:6d}  {ms:11.3f}  {pr:12.3f}  {100 * (pr - ms) / ms:+6.2f}%")
        for (l, _, _, ms, name), e in zip(vs, ve):
            lines.append(f"  {name:26s} {ms:11.3f}  {model.predict_lengths(l, H, D):12.3f}  {100 * e:+6.2f}%  (held out)")
        lines.append("")
    av = np.asarray(all_val)
    lines.append(f"All shapes, held-out packs: rms relative error {100 * float(np.sqrt(np.mean(av ** 2))):.2f}%, "
                 f"max {100 * float(np.max(np.abs(av))):.2f}%")
    # alpha_1: the block's linear operations, measured as GEMMs (not part of libt2vattn).
    gem = gemm_proxy_sweep()
    lines.append("")
    lines.append("alpha_1 of Eq. (9), measured: the linear operations of one DiT block (QKV d x 3d, output d x d, MLP "
                 "d x 4d and 4d x d), forward and backward (72 d^2 flops per token), as bf16 torch.matmul GEMMs:")
    lines.append("  hidden d   tokens   ms      TFLOP/s   -> alpha1_linear (ms/token)   c (ms)")
    models = {}
    for name, layers, H, D in TABLE2_MODELS:
        d = H * D
        a1, c1, tf, rows = gem[d]
        for n, ms in rows:
            lines.append(f"  {d:8d} {n:8d} {ms:8.3f} {72.0 * d * d * n / (ms * 1e-3) * 1e-12:9.0f}")
        lines.append(f"  {d:8d}  fit: alpha1_linear = {a1:.6e} ms/token, c = {c1:.4f} ms")
        fs = [x for x in fit_samples if x[1] == H and x[2] == D]
        model, _ = costmodel.fit(fs)
        models[name] = {"layers": layers, "heads": H, "head_dim": D, "hidden": d,
                        "alpha2_ms_per_token2": model.alpha2(H, D), "alpha1_attention_ms_per_token": model.alpha1(H, D),
                        "c0_attention_ms": model.c0, "alpha1_linear_ms_per_token": a1, "c_linear_ms": c1,
                        "gemm_tflops_at_65536_tokens": round(tf, 1)}
    lines.append("")
    lines.append("L_{c,k=1} per Table II model (one DiT cascade, fwd + bwd of all layers; k = 1, no communication):")
    lines.append("  L(B, S) = layers * ((alpha1_linear + alpha1_attention) * B*S + alpha2 * B*S^2)")
    for name, m in models.items():
        a1 = m["layers"] * (m["alpha1_linear_ms_per_token"] + m["alpha1_attention_ms_per_token"])
        a2 = m["layers"] * m["alpha2_ms_per_token2"]
        lines.append(f"  {name:17s} ({m['layers']} layers, {m['heads']} x {m['head_dim']}): alpha1 = {a1:.4e} ms/token, "
                     f"alpha2 = {a2:.4e} ms/token^2; e.g. one 20,280-token clip: {a1 * 20280 + a2 * 20280 ** 2:.0f} ms, "
                     f"attention share {100 * a2 * 20280 ** 2 / (a1 * 20280 + a2 * 20280 ** 2):.0f}%")
    with open(DIT_COST_FILE, "w") as f:
        json.dump({"kernel_source_hash": kernel_source_hash(), "models": models,
                   "note": "alpha2 and alpha1_attention: libt2vattn fwd+bwd per layer (fitted); alpha1_linear: the "
                           "block's GEMMs fwd+bwd per layer (torch.matmul, measured); written by bench.py --cost-model"},
                  f, indent=1, sort_keys=True)
    return "\n".join(lines)


def shares_report(seed: int = 0):
    """One GPU's share of a workload under k-way head sharding (Ulysses sequence parallelism,
    Section II-C: an All-to-All turns token sharding into head sharding, so each GPU runs
    attention over the full cu_seqlens at H / k heads). Times fwd+bwd of the library at each
    share shape, with the tile rows it chooses and with forced wide / narrow tiles, and the
    host scheduler's predicted makespan over its lower bound for the forward work list."""
    import numpy as np
    import torch

    from paper_2607_01701_amd import _lib
    from paper_2607_01701_amd.workload import workload_shape

    lines = ["Command (repo root, on the GPU): python3 bench.py --shares",
             f"Kernel source hash (bench.py kernel_source_hash): {kernel_source_hash()}", "",
             "One GPU's share under k-way head sharding: the workload's clips (seed 0) at H / k heads, D = 128,",
             "inputs N(0,1) in bf16 drawn on the GPU (torch generator, seed 1); the All-to-All itself is not run.",
             "TFLOP/s at 14 H D sum(L^2) per GPU; auto = the library's own tile choice; wide / narrow = forced",
             "256- / 128-query forward and dQ tiles (T2V_QTILE); LPT = host list-scheduling makespan / lower bound",
             "of the forward work list at the tile rows auto chose.", "",
             f"{'workload':9s} {'k':>2s} {'heads':>5s} {'auto ms':>9s} {'auto TF/s':>9s} {'fwd rows':>8s} {'fwd tiles':>9s} "
             f"{'wide TF/s':>9s} {'narrow TF/s':>11s} {'LPT':>6s}"]
    ncu = torch.cuda.get_device_properties(0).multi_processor_count

    def step(cu, q, k, v, g, scale, reps):
        for _ in range(2):
            o, lse = _lib.attn_fwd(q, k, v, cu, scale)
            _lib.attn_bwd(q, k, v, o, lse, g, cu, scale)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            o, lse = _lib.attn_fwd(q, k, v, cu, scale)
            _lib.attn_bwd(q, k, v, o, lse, g, cu, scale)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    for name, ks in (("long", (1, 2, 4, 8)), ("skew", (1, 2, 4, 8)), ("hetero", (1, 2, 4, 8))):
        _, lens, H, D = workload_shape(name, seed)
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        T = int(cu[-1])
        ssq = float(np.sum(np.asarray(lens, dtype=np.float64) ** 2))
        for kdeg in ks:
            h = H // kdeg
            gen = torch.Generator(device="cuda").manual_seed(1)
            q, k, v, g = (torch.randn(T, h, D, device="cuda", generator=gen).bfloat16() for _ in range(4))
            reps = 3 if name != "hetero" else 10
            flops = 14.0 * h * D * ssq
            res = {}
            for mode in ("auto", "wide", "narrow"):
                if mode == "auto":
                    os.environ.pop("T2V_QTILE", None)
                else:
                    os.environ["T2V_QTILE"] = mode
                res[mode] = step(cu, q, k, v, g, D ** -0.5, reps)
            os.environ.pop("T2V_QTILE", None)
            # The forward tile rows the library chose: one traced forward takes one record per item.
            n_wide = _lib.t2v_build_worklist(cu, h, 256, _lib.ORDER_LONGEST_FIRST).shape[0]
            n_narrow = _lib.t2v_build_worklist(cu, h, 128, _lib.ORDER_LONGEST_FIRST).shape[0]
            rec = torch.zeros(4 * max(n_wide, n_narrow), dtype=torch.int64, device="cuda")
            _lib.t2v_trace_set(rec.data_ptr(), max(n_wide, n_narrow))
            try:
                _lib.attn_fwd(q, k, v, cu, D ** -0.5)
                torch.cuda.synchronize()
                n_traced, _ = _lib.t2v_trace_count()
            finally:
                _lib.t2v_trace_set(None, 0)
            rows = 256 if n_traced == n_wide else 128
            items = _lib.t2v_build_worklist(cu, h, rows, _lib.ORDER_LONGEST_FIRST)
            mk, lb = _lib.t2v_plan_makespan(items, rows, ncu)
            lines.append(f"{name:9s} {kdeg:2d} {h:5d} {res['auto']:9.3f} {flops / res['auto'] * 1e-9:9.1f} "
                         f"{rows:8d} {items.shape[0]:9d} {flops / res['wide'] * 1e-9:9.1f} "
                         f"{flops / res['narrow'] * 1e-9:11.1f} {mk / lb:6.3f}")
            print(lines[-1], file=sys.stderr, flush=True)
            del q, k, v, g
            torch.cuda.empty_cache()
    return "\n".join(lines)


def balance_report(workload: str = "hetero", seed: int = 0):
    """Per-CU balance of each attention kernel on one traced fwd+bwd step, for both scheduler
    orders: per-CU busy time (summed workgroup durations from the library's workgroup trace),
    its coefficient of variation over the CUs (the single-GPU analogue of the per-rank CV of
    the paper's case study, Section V-E), and the idle share of CU time within the kernel's
    span; beside it the host scheduler's own predicted makespan over its lower bound."""
    import numpy as np
    import torch

    from paper_2607_01701_amd import _lib
    from paper_2607_01701_amd.workload import DESCRIPTIONS, make_workload

    pack = make_workload(workload, seed=seed)
    H, D, T = pack.heads, pack.head_dim, pack.total_tokens

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()

    q, k, v, g = dev(pack.q), dev(pack.k), dev(pack.v), dev(pack.dout)
    ncu = torch.cuda.get_device_properties(0).multi_processor_count
    lines = ["Command (repo root, on the GPU): python3 bench.py --balance",
             f"Kernel source hash (bench.py kernel_source_hash): {kernel_source_hash()}", "",
             f"Per-CU balance of one traced fwd+bwd step, {workload} workload ({DESCRIPTIONS[workload]}), "
             f"{ncu} CUs.",
             "busy = summed durations of the workgroups a CU ran; CV = std / mean of busy over the CUs; "
             "idle = 1 - sum(busy) / (CUs x kernel span);",
             "host LPT = the scheduler's predicted list-scheduling makespan over its lower bound "
             "(max(total / slots, largest item)) for the same work list.", "",
             f"{'order':14s} {'kernel':9s} {'WGs':>6s} {'CUs':>4s} {'span ms':>8s} {'busy mean ms':>12s} "
             f"{'CV':>6s} {'idle':>6s} {'host LPT':>9s}"]
    # Wide forward / dQ tiles and no dK/dV loop split (what the heterogeneous mix uses by
    # default), so that t2v_build_worklist reproduces the traced work lists.
    rows = {"fwd": 256, "bwd_dkdv": 128, "bwd_dq": 256}
    names = {0: "fwd", 2: "bwd_dkdv", 3: "bwd_dq"}
    os.environ["T2V_QTILE"], os.environ["T2V_SPLIT"] = "wide", "off"
    lines.insert(-2, "Tiles: 256 queries (forward, dQ), 128 keys (dK/dV), no loop split.")
    for order in ("longest_first", "natural"):
        os.environ["T2V_ORDER"] = order
        _lib.attn_fwd(q, k, v, pack.cu_seqlens, pack.scale)  # builds and caches the work lists
        cap = sum(_lib.t2v_build_worklist(pack.cu_seqlens, H, r,
                                          _lib.ORDER_NATURAL if order == "natural" else _lib.ORDER_LONGEST_FIRST
                                          ).shape[0] for r in rows.values())
        rec = torch.zeros(4 * cap, dtype=torch.int64, device="cuda")
        torch.cuda.synchronize()
        _lib.t2v_trace_set(rec.data_ptr(), cap)
        try:
            out, lse = _lib.attn_fwd(q, k, v, pack.cu_seqlens, pack.scale)
            _lib.attn_bwd(q, k, v, out, lse, g, pack.cu_seqlens, pack.scale)
            torch.cuda.synchronize()
            n, over = _lib.t2v_trace_count()
        finally:
            _lib.t2v_trace_set(None, 0)
        if n != cap or over:
            raise SystemExit(f"trace took {n} of {cap} records ({over} launches did not fit)")
        r = rec.view(cap, 4).cpu().numpy().astype(np.int64)
        for slot, name in names.items():
            x = r[r[:, 3] == slot]
            t0, t1 = x[:, 1], x[:, 2]
            span = float(t1.max() - t0.min())
            busy = {}
            for cu, d in zip(x[:, 0], t1 - t0):
                busy[cu] = busy.get(cu, 0) + int(d)
            b = np.array(list(busy.values()), dtype=np.float64)
            b = np.concatenate([b, np.zeros(max(0, ncu - len(b)))])  # CUs that ran nothing
            items = _lib.t2v_build_worklist(pack.cu_seqlens, H, rows[name],
                                            _lib.ORDER_NATURAL if order == "natural" else _lib.ORDER_LONGEST_FIRST)
            mk, lb = _lib.t2v_plan_makespan(items, rows[name], ncu)
            lines.append(f"{order:14s} {name:9s} {x.shape[0]:6d} {len(busy):4d} {span * 1e-5:8.3f} "
                         f"{b.mean() * 1e-5:12.3f} {b.std() / b.mean():6.3f} {1 - b.sum() / (ncu * span):6.1%} "
                         f"{mk / lb:9.3f}")
    for var in ("T2V_ORDER", "T2V_QTILE", "T2V_SPLIT"):
        os.environ.pop(var, None)
    lines += ["", "(device clock 100 MHz: 1 tick = 10 ns)"]
    return "\n".join(lines)


def plan_batch_report(n_gpus: int = 16, seed: int = 0):
    """Cascade plan of one batch (paper Section IV-A, Eqs. (1)-(7); Alg. 1) on the CPU.

    Each clip of the heterogeneous mix is three cascades: VAE encode -> DiT forward/backward,
    and a text encoder -> the same DiT cascade. The DiT's latency at degree k follows Eq. (9):
    (alpha_1 S + alpha_2 S^2) / k over 60 layers (HunyuanVideo-13B shape, 24 x 128), with alpha_2
    and the attention's per-token term fitted to libt2vattn and alpha_1 of the block's linear
    operations measured as bf16 GEMMs (both by --cost-model on the GPU), plus an All-to-All
    term for k > 1 over xGMI; memory follows Eq. (8). The VAE and text-encoder latencies are
    linear in tokens. Every constant not measured is stated below and is an assumption of
    this synthetic batch, not a measurement.
    """
    import numpy as np

    from paper_2607_01701_amd import planner
    from paper_2607_01701_amd.workload import workload_shape

    lengths = workload_shape("hetero", seed)[1]
    # Measured coefficients (bench.py --cost-model on the GPU, profiles/dit_cost_model.json):
    # attention alpha_2 and its per-token term from libt2vattn, alpha_1 of the block's linear
    # operations from the GEMM proxy; per layer, fwd + bwd, in ms.
    with open(DIT_COST_FILE) as f:
        m = json.load(f)["models"]["HunyuanVideo-13B"]
    layers, H, D = m["layers"], m["heads"], m["head_dim"]
    alpha2 = m["alpha2_ms_per_token2"] * 1e-3 * layers                # s per token^2, all layers
    alpha1_attn = m["alpha1_attention_ms_per_token"] * 1e-3 * layers  # s per token
    alpha1_rest = m["alpha1_linear_ms_per_token"] * 1e-3 * layers      # s per token: the block's GEMMs
    hidden_bytes = H * D * 2
    a2a_bw = 7 * 153e9                           # xGMI: 7 links x ~153 GB/s per GPU
    W = 288e9                                    # bytes per GPU
    mem_states = 13e9 * 16 / n_gpus + 8e9        # ZeRO-3 sharded model states + workspace (assumption)
    mem_token = 60 * hidden_bytes * 34           # activation bytes per token across the layers (assumption)
    K = [k for k in (1, 2, 4, 8) if k <= n_gpus]
    preds, lat, mem, names = [], [], [], []
    for i, S in enumerate(lengths):
        v = len(preds)                            # VAE encode of the clip
        preds.append([])
        lat.append([S * 2.0e-6 / k ** 0.9 for k in K])
        mem.append([20e9 + S * 4.0e5 / k for k in K])
        names.append(f"vae{i}")
        t = len(preds)                            # text encoder (short sequence)
        preds.append([])
        lat.append([0.02 / k ** 0.5 for k in K])
        mem.append([10e9] * len(K))
        names.append(f"txt{i}")
        preds.append([v, t])                      # DiT forward + backward
        comp = alpha1_attn * S + alpha2 * S * S + alpha1_rest * S
        lat.append([comp / k + (0.0 if k == 1 else 4 * layers * 2 * S * hidden_bytes * (k - 1) / k / a2a_bw)
                    for k in K])
        mem.append([mem_states + S * mem_token / k for k in K])
        names.append(f"dit{i}")
    n = len(preds)
    t0 = time.perf_counter()
    deg, starts, T = planner.plan(preds, K, lat, mem, W, n_gpus, population=64, generations=300, seed=seed)
    t_plan = time.perf_counter() - t0
    lines = ["Command (repo root, CPU only): python3 bench.py --plan", "",
             f"Cascade plan of one batch: the heterogeneous mix (seed {seed}, {len(lengths)} clips) as {n} cascades "
             f"on N = {n_gpus} GPUs, degrees K = {K} (Section IV-A, Eqs. (1)-(7); Alg. 1).",
             "Latency inputs, measured on one MI355X (profiles/dit_cost_model.json, HunyuanVideo-13B shape: "
             f"{layers} layers, {H} x {D}): attention alpha2 = {alpha2:.3e} s/token^2 and {alpha1_attn:.3e} s/token "
             f"(libt2vattn), the block's linear operations alpha1 = {alpha1_rest:.3e} s/token (bf16 GEMM proxy); "
             "assumed: All-to-All over 7 x 153 GB/s xGMI, VAE 2e-6 s/token / k^0.9, text encoder 0.02 s / k^0.5; "
             "memory Eq. (8) with assumed constants, W = 288 GB.",
             f"GA: population 64, 300 generations, planning time {t_plan:.2f} s (host CPU, one thread).",
             f"Planned makespan: {T:.2f} s", "", "Static parallel degree for every cascade (list-scheduled, same DAG):"]
    for k in K:
        j = K.index(k)
        if all(mem[c][j] <= W for c in range(n)):
            _, Tk = planner.list_schedule(preds, [k] * n, [lat[c][j] for c in range(n)], n_gpus)
            lines.append(f"  k = {k}: {Tk:.2f} s  (the plan is {100 * (1 - T / Tk):.1f}% shorter)")
        else:
            lines.append(f"  k = {k}: infeasible (memory)")
    lines.append("")
    lines.append("DiT cascades: clip tokens -> planned degree, start, end (s)")
    for c in range(n):
        if names[c].startswith("dit"):
            i = int(names[c][3:])
            lines.append(f"  {lengths[i]:6d}  k={deg[c]}  {starts[c]:8.2f}  {starts[c] + lat[c][K.index(deg[c])]:8.2f}")
    return "\n".join(lines)


def mfma_probe(blocks: int = 2048, iters: int = 40000) -> dict:
    """The library's MFMA throughput probe: bf16 dense TFLOP/s and shader clock this GPU
    sustains under a pure MFMA load (context for the attention kernels' rates)."""
    import torch

    from paper_2607_01701_amd import _lib

    _lib.lib()
    rec = torch.zeros(3 * blocks, dtype=torch.int64, device="cuda")
    stream = torch.cuda.current_stream().cuda_stream
    _lib.t2v_probe_mfma_peak(rec.data_ptr(), blocks, 2000, stream)  # warm-up
    r = _lib.t2v_probe_mfma_peak(rec.data_ptr(), blocks, iters, stream)
    print(f"[bench] MFMA probe: {r['tflops']:.0f} TFLOP/s at {r['ghz']:.2f} GHz", file=sys.stderr, flush=True)
    return {"tflops": round(r["tflops"], 1), "ghz": round(r["ghz"], 3), "ms": round(r["ms"], 3),
            "frac_of_spec_peak": round(r["tflops"] / PEAK_BF16_TFLOPS, 4),
            "kernel": "4 waves x 4 independent v_mfma_f32_32x32x16_bf16 chains per workgroup, "
                      f"{blocks} workgroups x {iters} rounds"}


def device_normal(shape, gen):
    """bf16 N(0,1) values drawn on the GPU from a seeded generator (timing-only inputs)."""
    import torch
    return torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)


def run_workload(workload, seed, steps, warmup, order=None, device_values=False):
    """Times `steps` fwd+bwd steps of one workload after `warmup` untimed ones; returns the
    bench record (without the CPU baseline) and the pack.

    device_values: draw the N(0,1) inputs on the GPU (seeded) instead of on the host; the
    timing-only summaries of the other workloads use this, since drawing the largest packs
    on the host takes longer than timing them."""
    import numpy as np
    import torch

    from paper_2607_01701_amd import _lib
    from paper_2607_01701_amd.workload import DESCRIPTIONS, attention_flops, make_workload

    if order is not None:
        os.environ["T2V_ORDER"] = order  # read by the library at each call
    t_gen = time.perf_counter()
    pack = make_workload(workload, seed=seed, tensors=not device_values)
    H, D, T = pack.heads, pack.head_dim, pack.total_tokens
    print(f"[bench] workload {workload}: T={T} H={H} D={D} sum(Lq*Lk)={pack.sum_qk} "
          f"(generated in {time.perf_counter() - t_gen:.1f}s)", file=sys.stderr, flush=True)

    def dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()

    if device_values:
        gen = torch.Generator(device="cuda").manual_seed(seed)
        Tk = pack.total_tokens_k if pack.cu_seqlens_k is not None else T
        q, k, v, g = (device_normal((n, H, D), gen) for n in (T, Tk, Tk, T))
    else:
        q, k, v, g = dev(pack.q), dev(pack.k), dev(pack.v), dev(pack.dout)
    out = torch.empty_like(q)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(k)
    lse = torch.empty((H, T), dtype=torch.float32, device="cuda")
    delta = torch.empty((2, H, T), dtype=torch.float32, device="cuda")
    cu = np.ascontiguousarray(pack.cu_seqlens, dtype=np.int32)
    cross = pack.cu_seqlens_k is not None
    cuk = np.ascontiguousarray(pack.cu_seqlens_k if cross else pack.cu_seqlens, dtype=np.int32)
    cukp = cuk.ctypes.data_as(_lib._i32p)
    nseq = cu.shape[0] - 1
    L = _lib.lib()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    cup = cu.ctypes.data_as(_lib._i32p)

    def step(mid=None):
        if cross:
            st = L.t2v_attn_fwd_qk(q.data_ptr(), k.data_ptr(), v.data_ptr(), cup, cukp, nseq, H, D, pack.scale,
                                   out.data_ptr(), lse.data_ptr(), sh)
        else:
            st = L.t2v_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cup, nseq, H, D, pack.scale,
                                out.data_ptr(), lse.data_ptr(), sh)
        if st:
            raise _lib.T2VError(st, _lib.t2v_last_error())
        if mid is not None:
            mid.record(stream)
        if cross:
            st = L.t2v_attn_bwd_qk(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(), cup, cukp,
                                   nseq, H, D, pack.scale, g.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                   delta.data_ptr(), sh)
        else:
            st = L.t2v_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(), cup, nseq,
                                H, D, pack.scale, g.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                delta.data_ptr(), sh)
        if st:
            raise _lib.T2VError(st, _lib.t2v_last_error())

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup {warmup} steps done", file=sys.stderr, flush=True)

    _lib.t2v_timing_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # Per step: events before the forward, between forward and backward, after the backward.
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(steps):
        marks[i][0].record(stream)
        step(marks[i][1])
        marks[i][2].record(stream)
    e1.record(stream)
    torch.cuda.synchronize()
    ktimes = _lib.t2v_kernel_times()
    _lib.t2v_timing_enable(False)
    ms_step = e0.elapsed_time(e1) / steps
    print(f"[bench] timed {steps} steps: {ms_step:.3f} ms/step", file=sys.stderr, flush=True)
    per = {"fwd": [m[0].elapsed_time(m[1]) for m in marks], "bwd": [m[1].elapsed_time(m[2]) for m in marks],
           "fwd_bwd": [m[0].elapsed_time(m[2]) for m in marks]}

    fl = attention_flops(pack)
    tflops = fl["fwd_bwd"] / (ms_step * 1e-3) * 1e-12
    avg = {name: (ms / n if n else None) for name, (ms, n) in ktimes.items()}
    kf = kernel_flops(H, D, pack.sum_qk)
    kernels = {}
    for name, a in avg.items():
        entry = {"avg_ms": a, "launches": ktimes[name][1]}
        if a and name in kf:
            entry["tflops"] = kf[name] / (a * 1e-3) * 1e-12
        if a and name == "bwd_pre":
            # out and dout read (4 D bytes per (token, head)), lse read, -Delta and lse2 written
            entry["gbs"] = (4.0 * T * H * D + 12.0 * T * H) / (a * 1e-3) * 1e-9
        kernels[name] = entry
    dominant = max((n for n in kf if avg.get(n)), key=lambda n: ktimes[n][0])
    achieved = kernels[dominant]["tflops"]
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        if rec.get("kernel_source_hash") == kernel_source_hash() and rec.get("workload") == workload:
            traffic = rec.get("kernels", {}).get(dominant, {}).get("hbm_bytes_per_launch")
    roofline = {"bound": "mfma", "kernel": dominant, "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": traffic,
                "algorithmic_per_launch": kf[dominant],
                "algorithmic_note": {"fwd": "4*H*D*sum(L^2)", "bwd_dkdv": "8*H*D*sum(L^2)",
                                     "bwd_dq": "6*H*D*sum(L^2)"}[dominant]}
    fwd_ms = avg["fwd"]
    bwd_ms = sum(avg[n] for n in ("bwd_pre", "bwd_dkdv", "bwd_dq") if avg.get(n))
    conv = {"fwd": fl["fwd"], "bwd": fl["bwd"], "fwd_bwd": fl["fwd_bwd"]}
    timing = {}
    for name, xs in per.items():
        med = float(np.median(xs))
        timing[name] = {"median_ms": round(med, 4), "mean_ms": round(float(np.mean(xs)), 4),
                        "min_ms": round(float(np.min(xs)), 4),
                        "tflops_at_median": round(conv[name] / (med * 1e-3) * 1e-12, 2)}
    flops = {"counted_fwd_bwd": fl["fwd_bwd"], "strict_no_recompute": fl["no_recompute"],
             "executed_mfma": fl["executed"],
             "tflops_strict_no_recompute": round(fl["no_recompute"] / (ms_step * 1e-3) * 1e-12, 2),
             "tflops_executed_mfma": round(fl["executed"] / (ms_step * 1e-3) * 1e-12, 2),
             "exp2_fwd": H * pack.sum_qk, "exp2_bwd": 2 * H * pack.sum_qk,
             "note": "counted 14, strict no-recompute 12, executed 18 (fwd 4 + dK/dV 8 + dQ 6) x H*D*sum(Lq*Lk)"}
    res = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: seeded N(0,1) values rounded to bf16; clip lengths from latent grids (no dataset)",
        "config": {"workload": f"{workload}: {DESCRIPTIONS[workload]}", "seed": seed,
                   "total_tokens": T, "heads": H, "head_dim": D, "sum_sq_len": pack.sum_qk,
                   "clip_lengths": pack.lengths.tolist() if pack.nseq <= 32 else f"{pack.nseq} clips",
                   "flop_convention": "fwd 4*H*D*sum(Lq*Lk) + bwd 10*H*D*sum(Lq*Lk) (Lq = Lk = L for "
                                      "self-attention)"},
        "frac_of_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "fwd_tflops": round(fl["fwd"] / (fwd_ms * 1e-3) * 1e-12, 2),
        "bwd_tflops": round(fl["bwd"] / (bwd_ms * 1e-3) * 1e-12, 2),
        "timing": timing,
        "flops": flops,
        "kernels": kernels,
        "roofline": roofline,
        "kernel_source_hash": kernel_source_hash(),
    }
    if cross:
        res["config"]["key_lengths"] = pack.lengths_k.tolist() if pack.nseq <= 32 else f"{pack.nseq} sequences"
        res["config"]["total_tokens_k"] = pack.total_tokens_k
    if order is not None:
        res["config"]["scheduler_order"] = order
    del q, k, v, g, out, dq, dk, dv, lse, delta
    torch.cuda.empty_cache()
    return res, pack


# The default line's summary of every workload: (name, timed steps, warmup steps). The long
# and skewed packs take 0.26 and 0.77 s per step, so they get few.
WORKLOAD_STEPS = (("tiny", 50, 10), ("uniform", 20, 5), ("long", 4, 1), ("skew", 3, 1))


def workloads_summary(seed: int, main_res: dict) -> dict:
    """fwd and fwd+bwd TFLOP/s, fraction of the bf16 peak and ms per step of the five workloads
    (the heterogeneous mix from the headline run, the others timed here with inputs drawn on
    the GPU)."""
    out = {}

    def entry(r, steps):
        return {"fwd_bwd_tflops": r["value"], "frac_of_peak": r["frac_of_peak"], "fwd_tflops": r["fwd_tflops"],
                "fwd_frac_of_peak": round(r["fwd_tflops"] / PEAK_BF16_TFLOPS, 4), "ms_per_step": r["ms_per_step"],
                "fwd_ms": r["timing"]["fwd"]["median_ms"], "steps": steps,
                "config": r["config"]["workload"], "sum_sq_len": r["config"]["sum_sq_len"]}

    for name, steps, warmup in WORKLOAD_STEPS[:2]:
        r, _ = run_workload(name, seed, steps, warmup, device_values=True)
        out[name] = entry(r, steps)
    out["hetero"] = entry(main_res, main_res["steps"])
    for name, steps, warmup in WORKLOAD_STEPS[2:]:
        r, _ = run_workload(name, seed, steps, warmup, device_values=True)
        out[name] = entry(r, steps)
    return out


def fresh_pack_report(seed: int = 0, n_base: int = 16, steps: int = 32) -> dict:
    """Cost of a new cu_seqlens on every call (clip lengths change from batch to batch,
    Section III, Observation 1) against the cached-plan path, on the same GPU work.

    Base packs: the heterogeneous mix at seeds seed .. seed + n_base - 1. Cached: the steps
    cycle over the base packs, whose work lists (3 per pack, 48 in all) stay in the library's
    cache. Fresh: each step takes the next base pack with its clips in a new random order, a
    cu_seqlens the library has not seen, so every call builds, uploads and caches new work
    lists and, past 64 lists, releases old ones. Both runs do the same clips per step, so
    the difference is the cache-miss cost as the GPU sees it."""
    import numpy as np
    import torch

    from paper_2607_01701_amd import _lib
    from paper_2607_01701_amd.workload import cu_from_lengths, workload_shape

    base = [list(workload_shape("hetero", seed + i)[1]) for i in range(n_base)]
    _, _, H, D = workload_shape("hetero", seed)
    tmax = max(sum(b) for b in base)
    gen = torch.Generator(device="cuda").manual_seed(seed + 7)
    q, k, v, g = (device_normal((tmax, H, D), gen) for _ in range(4))
    out, dq, dk, dv = (torch.empty_like(q) for _ in range(4))
    lse = torch.empty((H, tmax), dtype=torch.float32, device="cuda")
    ws = torch.empty((2, H, tmax), dtype=torch.float32, device="cuda")
    L = _lib.lib()
    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    sc = 1.0 / D ** 0.5
    rng = np.random.default_rng(seed + 11)
    seen = set()

    def step(lengths):
        cu = np.ascontiguousarray(cu_from_lengths(lengths), dtype=np.int32)
        cup = cu.ctypes.data_as(_lib._i32p)
        st = L.t2v_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), cup, len(lengths), H, D, sc, out.data_ptr(),
                            lse.data_ptr(), sh)
        if st == 0:
            st = L.t2v_attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(), cup,
                                len(lengths), H, D, sc, g.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                ws.data_ptr(), sh)
        if st:
            raise _lib.T2VError(st, _lib.t2v_last_error())

    def fresh(i):
        while True:
            b = base[i % n_base]
            perm = [b[j] for j in rng.permutation(len(b))]
            if tuple(perm) not in seen and perm != b:
                seen.add(tuple(perm))
                return perm

    def timed(lengths_of):
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        h0 = time.perf_counter()
        e0.record(stream)
        for i in range(steps):
            step(lengths_of(i))
        e1.record(stream)
        host_ms = (time.perf_counter() - h0) * 1e3 / steps
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps, host_ms

    _lib.t2v_release_cache()
    for b in base:  # cached: every base pack's three work lists built once
        step(b)
    for i in range(3):
        step(fresh(i))
    cached_ms, cached_host = timed(lambda i: base[i % n_base])
    fresh_ms, fresh_host = timed(lambda i: fresh(i))
    ssq = sum(sum(x * x for x in base[i % n_base]) for i in range(steps)) / steps
    fl = 14.0 * H * D * ssq
    del q, k, v, g, out, dq, dk, dv, lse, ws
    torch.cuda.empty_cache()
    res = {"cached_ms_per_step": round(cached_ms, 4), "fresh_ms_per_step": round(fresh_ms, 4),
           "cached_tflops": round(fl / (cached_ms * 1e-3) * 1e-12, 2),
           "fresh_tflops": round(fl / (fresh_ms * 1e-3) * 1e-12, 2),
           "overhead_pct": round(100.0 * (fresh_ms / cached_ms - 1.0), 2),
           "host_ms_per_call_pair": {"cached": round(cached_host, 3), "fresh": round(fresh_host, 3)},
           "steps": steps,
           "packs": f"hetero mix, seeds {seed}..{seed + n_base - 1}; fresh steps permute a base pack's clip order "
                    f"(new cu_seqlens every call: 3 new work lists per fwd+bwd, 64 cached)"}
    print(f"[bench] fresh packs: cached {cached_ms:.3f} ms/step, fresh {fresh_ms:.3f} ms/step "
          f"({res['overhead_pct']:+.2f}%)", file=sys.stderr, flush=True)
    return res


def main():
    args = parse_args()
    if args.ingest_rocpd:
        ingest_rocpd(*args.ingest_rocpd, workload=args.workload)
        return
    if args.ingest_mfma:
        ingest_mfma(args.ingest_mfma, workload=args.workload)
        return
    if args.ingest_sq:
        ingest_sq(args.ingest_sq, workload=args.workload)
        return
    if args.write_summaries:
        write_summaries(*args.write_summaries[:2])
        return
    if args.plan:
        print(plan_batch_report(), flush=True)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): libt2vattn "
              "has no multi-GPU path; sharding across GPUs is not implemented.", file=sys.stderr, flush=True)
        sys.exit(2)
    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration()
        return

    if args.cost_model:
        print(cost_model_sweep(), flush=True)
        return
    if args.balance:
        print(balance_report(args.workload, args.seed), flush=True)
        return
    if args.shares:
        print(shares_report(args.seed), flush=True)
        return
    if args.sweep:
        # Smaller step counts for the long workloads keep the sweep to about a minute of GPU time.
        lf = "longest_first"
        plan = [("tiny", lf, 50), ("uniform", lf, 20), ("hetero", lf, 20), ("long", lf, 5), ("skew", lf, 3), ("cross", lf, 20),
                ("hetero", "natural", 20), ("skew", "natural", 3)]
        for name, order, steps in plan:
            res, _ = run_workload(name, args.seed, steps, max(1, min(args.warmup, steps // 2)), order)
            print(json.dumps(res), flush=True)
        return
    res, pack = run_workload(args.workload, args.seed, args.steps, args.warmup)
    res["mfma_probe"] = mfma_probe()
    res["roofline"]["frac_of_probe"] = round(res["roofline"]["achieved"] / res["mfma_probe"]["tflops"], 4)
    # The step against the MFMA ceiling measured on this GPU (context beside the published peak).
    res["frac_of_probe_peak"] = round(res["value"] / res["mfma_probe"]["tflops"], 4)
    if args.workload == "hetero" and not args.no_extras:
        res["workloads"] = workloads_summary(args.seed, res)
        res["fresh_packs"] = fresh_pack_report(args.seed)
        res["paper_context"] = PAPER_CONTEXT
    if not args.no_cpu_baseline:
        print("[bench] timing the float64 oracle on a bounded sample", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(pack)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
