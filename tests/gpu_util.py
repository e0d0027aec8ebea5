"""Helpers for GPU tests: move seeded packs to the device, run the HIP path, compare."""
import sys
import time

import numpy as np

TOL_REL = 2e-2   # out, dq, dk, dv: max |gpu - ref| / max |ref|
TOL_LSE = 1e-3   # lse: max |gpu - ref| (natural log)


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


def to_dev(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_inputs(pack):
    return {n: to_dev(getattr(pack, n)) for n in ("q", "k", "v", "dout")}


def run_hip(pack, dev=None, scale=None):
    """fwd + bwd through the C ABI; returns device tensors."""
    import torch
    from paper_2607_01701_amd import attn_bwd, attn_fwd
    d = dev_inputs(pack) if dev is None else dev
    sc = pack.scale if scale is None else scale
    ck = pack.cu_seqlens_k
    out, lse = attn_fwd(d["q"], d["k"], d["v"], pack.cu_seqlens, sc, cu_seqlens_k=ck)
    dq, dk, dv = attn_bwd(d["q"], d["k"], d["v"], out, lse, d["dout"], pack.cu_seqlens, sc, cu_seqlens_k=ck)
    torch.cuda.synchronize()
    return {"out": out, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def to_np(res):
    return {k: v.float().cpu().numpy().astype(np.float64) for k, v in res.items()}


def rel_err(g, r):
    den = float(np.max(np.abs(r)))
    return float(np.max(np.abs(g - r))) / den if den > 0 else float(np.max(np.abs(g)))


def compare_full(g, ref, cu, label="", cu_k=None):
    """Whole-tensor gate plus a per-sequence diagnostic (dk, dv on the key offsets cu_k when
    given). Returns dict of errors."""
    cu_k = cu if cu_k is None else cu_k
    errs = {k: rel_err(g[k], ref[k]) for k in ("out", "dq", "dk", "dv")}
    errs["lse"] = float(np.max(np.abs(g["lse"] - ref["lse"]))) if g["lse"].size else 0.0
    worst = {}
    for s in range(len(cu) - 1):
        for k in ("out", "dq", "dk", "dv"):
            c = cu if k in ("out", "dq") else cu_k
            a, b = int(c[s]), int(c[s + 1])
            if b == a:
                continue
            e = rel_err(g[k][a:b], ref[k][a:b])
            worst[k] = max(worst.get(k, 0.0), e)
    log(f"{label} errors {errs} worst-per-clip {worst}")
    return errs, worst


def assert_within(errs):
    for k in ("out", "dq", "dk", "dv"):
        assert errs[k] <= TOL_REL, f"{k} relative max error {errs[k]:.3e} > {TOL_REL}"
    assert errs["lse"] <= TOL_LSE, f"lse abs error {errs['lse']:.3e} > {TOL_LSE}"
