"""Parity at the full sizes of the four large workloads, in the launch configuration the
benchmark times (same entry points, same work lists, default scheduler order).

The tolerance gate (relative max error over the whole packed tensor, 2e-2 for out, dq, dk,
dv; 1e-3 absolute for lse) is computed on:
* uniform: the full oracle, every clip and head, whole tensors;
* hetero: the full oracle on the head subset {0, H/2, H-1} over every clip (heads are
  independent, so the subset is exact for those heads), whole tensors restricted to them,
  plus the per-clip errors, each held to the same bound;
* long and skew (75,600- and 100,800-token clips, where one head alone is ~10^10 scores):
  dk and dv for every key of one head of the long clip (the oracle forms that head's whole
  backward), out / lse / dq at sampled rows of every head, and the complete outputs of the
  short clips.
Properties that hold at any size are checked for every (clip, head): sum_j dk_j = 0,
sum_j dv_j = sum_i dout_i, <Q, dQ> = <K, dK>.
"""
import numpy as np
import pytest

import oracle
from paper_2607_01701_amd.workload import bf16_bits_to_f32, make_workload

from gpu_util import TOL_LSE, TOL_REL, log, run_hip

pytestmark = pytest.mark.gpu

_CACHE = {}


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    _CACHE.clear()
    torch.cuda.empty_cache()


def workload_run(name):
    """Inputs (host bf16 bits) and the HIP outputs (device tensors) of a workload, once per module."""
    if name not in _CACHE:
        _CACHE.clear()
        log(f"generating {name}")
        pack = make_workload(name)
        log(f"running fwd+bwd on {name}: T={pack.total_tokens} H={pack.heads} D={pack.head_dim}")
        res = run_hip(pack)
        _CACHE[name] = (pack, res)
    return _CACHE[name]


def f64(bits):
    return bf16_bits_to_f32(bits).astype(np.float64)


def gpu_rows(t, tokens, heads):
    """Selected (token, head) rows of a device [T, H, D] tensor, as float64."""
    import torch
    ti = torch.as_tensor(np.asarray(tokens), device=t.device)
    hi = torch.as_tensor(np.asarray(heads), device=t.device)
    return t[ti, hi].double().cpu().numpy()


def sample_rows(pack, n_random=24, seed=1):
    """Clip boundaries, tile boundaries and random rows, over a spread of heads."""
    rng = np.random.default_rng(seed)
    cu = pack.cu_seqlens
    toks, hs = [], []
    clips = [s for s in range(pack.nseq) if cu[s + 1] > cu[s]]
    pick = clips if len(clips) <= 6 else list(rng.choice(clips, 6, replace=False))
    for s in pick:
        a, b = int(cu[s]), int(cu[s + 1])
        for t in (a, a + 1, min(b - 1, a + 127), min(b - 1, a + 128), min(b - 1, a + 255), b - 2, b - 1):
            if a <= t < b:
                toks.append(t)
                hs.append(int(rng.integers(pack.heads)))
    toks += list(rng.integers(0, pack.total_tokens, n_random))
    hs += list(rng.integers(0, pack.heads, n_random))
    return toks, hs


def slice_head(pack, name, a, b, h):
    return f64(getattr(pack, name)[a:b, h])


def check_query_rows(name):
    pack, res = workload_run(name)
    toks, hs = sample_rows(pack)
    log(f"{name}: oracle on {len(toks)} sampled query rows")
    cu = pack.cu_seqlens
    # The oracle reads each sampled row's clip for that head only.
    ref = {"out": [], "lse": [], "dq": []}
    slices = {}
    for t, h in zip(toks, hs):
        s = int(np.searchsorted(cu, t, side="right") - 1)
        a, b = int(cu[s]), int(cu[s + 1])
        if (s, h) not in slices:
            slices[(s, h)] = {n: slice_head(pack, n, a, b, h)[:, None, :] for n in ("q", "k", "v", "dout")}
        sl = slices[(s, h)]
        r = oracle.query_rows(sl["q"], sl["k"], sl["v"], sl["dout"], np.array([0, b - a]), pack.scale,
                              [t - a], [0])
        for key in ref:
            ref[key].append(r[key][0])
    ref = {k: np.asarray(v) for k, v in ref.items()}
    got_out = gpu_rows(res["out"], toks, hs)
    got_dq = gpu_rows(res["dq"], toks, hs)
    got_lse = res["lse"][np.asarray(hs), np.asarray(toks)].double().cpu().numpy()
    e_out = np.max(np.abs(got_out - ref["out"])) / np.max(np.abs(ref["out"]))
    e_dq = np.max(np.abs(got_dq - ref["dq"])) / np.max(np.abs(ref["dq"]))
    e_lse = np.max(np.abs(got_lse - ref["lse"]))
    log(f"{name}: sampled rows out {e_out:.3e} dq {e_dq:.3e} lse {e_lse:.3e}")
    assert e_out <= TOL_REL and e_dq <= TOL_REL and e_lse <= TOL_LSE


def check_full_oracle(name, heads=None):
    """The whole-tensor gate against the full oracle (all heads, or a head subset over every
    clip), with the per-clip errors logged and held to the same bound."""
    from gpu_util import compare_full
    pack, res = workload_run(name)
    hs = list(range(pack.heads)) if heads is None else list(heads)
    log(f"{name}: full oracle on every clip, heads {hs if heads is not None else 'all'}")
    sl = {n: f64(getattr(pack, n)[:, hs]) for n in ("q", "k", "v", "dout")}
    ref = oracle.attention(sl["q"], sl["k"], sl["v"], sl["dout"], pack.cu_seqlens, pack.scale)
    hidx = np.asarray(hs)
    got = {k: res[k][:, hidx].double().cpu().numpy() for k in ("out", "dq", "dk", "dv")}
    got["lse"] = res["lse"][hidx].double().cpu().numpy()
    errs, worst = compare_full(got, ref, pack.cu_seqlens, label=f"{name} heads {len(hs)}")
    for k in ("out", "dq", "dk", "dv"):
        assert errs[k] <= TOL_REL, (k, errs[k])
        assert worst[k] <= TOL_REL, (k, "per clip", worst[k])
    assert errs["lse"] <= TOL_LSE, errs["lse"]


def check_key_rows(name, seq, head, nkeys=12, torch_backend=False):
    """dk / dv of one (clip, head) at sampled keys, or at every key (nkeys=None)."""
    pack, res = workload_run(name)
    cu = pack.cu_seqlens
    a, b = int(cu[seq]), int(cu[seq + 1])
    L = b - a
    rng = np.random.default_rng(2)
    if nkeys is None:
        keys = list(range(L))
    else:
        keys = sorted(set([0, 1, 127, 128, L - 2, L - 1] + list(rng.integers(0, L, nkeys))))
    log(f"{name}: oracle dk/dv on clip {seq} (L={L}) head {head}, {len(keys)} keys")
    sl = {n: slice_head(pack, n, a, b, head)[:, None, :] for n in ("q", "k", "v", "dout")}
    if torch_backend:
        step = max(1, L // 8)

        def progress(r1, n):
            if r1 // step != (r1 - 2048) // step or r1 == n:
                log(f"{name}: oracle query rows {r1}/{n}")

        ref = oracle.key_rows_torch(sl["q"], sl["k"], sl["v"], sl["dout"], np.array([0, L]), pack.scale, 0, 0, keys,
                                    progress=progress)
    else:
        ref = oracle.key_rows(sl["q"], sl["k"], sl["v"], sl["dout"], np.array([0, L]), pack.scale, 0, 0, keys)
    toks = [a + j for j in keys]
    hs = [head] * len(keys)
    e_dk = np.max(np.abs(gpu_rows(res["dk"], toks, hs) - ref["dk"])) / np.max(np.abs(ref["dk"]))
    e_dv = np.max(np.abs(gpu_rows(res["dv"], toks, hs) - ref["dv"])) / np.max(np.abs(ref["dv"]))
    log(f"{name}: {'all' if nkeys is None else 'sampled'} keys dk {e_dk:.3e} dv {e_dv:.3e}")
    assert e_dk <= TOL_REL and e_dv <= TOL_REL


def check_short_clips(name, max_len, max_clips=2, heads=None):
    """Complete outputs of short clips (all heads unless given) against the full oracle."""
    pack, res = workload_run(name)
    cu = pack.cu_seqlens
    clips = [s for s in range(pack.nseq) if 0 < cu[s + 1] - cu[s] <= max_len][:max_clips]
    assert clips, "workload has no short clip"
    hs = list(range(pack.heads)) if heads is None else heads
    for s in clips:
        a, b = int(cu[s]), int(cu[s + 1])
        log(f"{name}: full oracle on clip {s} (L={b - a}) heads {len(hs)}")
        sl = {n: f64(getattr(pack, n)[a:b][:, hs]) for n in ("q", "k", "v", "dout")}
        ref = oracle.attention(sl["q"], sl["k"], sl["v"], sl["dout"], np.array([0, b - a]), pack.scale)
        hidx = np.asarray(hs)
        for key in ("out", "dq", "dk", "dv"):
            g = res[key][a:b][:, hidx].double().cpu().numpy()
            e = np.max(np.abs(g - ref[key])) / np.max(np.abs(ref[key]))
            assert e <= TOL_REL, (key, e)
        gl = res["lse"][hidx, a:b].double().cpu().numpy()
        assert np.max(np.abs(gl - ref["lse"])) <= TOL_LSE


def check_invariants(name):
    """P6, P7, P8 per (clip, head), in float64 on the device."""
    import torch
    pack, res = workload_run(name)
    cu = pack.cu_seqlens
    worst = {"sum_dk": 0.0, "sum_dv": 0.0, "qdq_kdk": 0.0}
    qd, kd, gd = (torch.from_numpy(np.ascontiguousarray(getattr(pack, n)).view(np.int16)).view(torch.bfloat16)
                  .cuda() for n in ("q", "k", "dout"))
    for s in range(pack.nseq):
        a, b = int(cu[s]), int(cu[s + 1])
        if b == a:
            continue
        dk = res["dk"][a:b].double()
        dv = res["dv"][a:b].double()
        dq = res["dq"][a:b].double()
        q, k, g = qd[a:b].double(), kd[a:b].double(), gd[a:b].double()
        # sum over keys vs the sum of magnitudes (per head and dim)
        r6 = (dk.sum(0).abs() / dk.abs().sum(0).clamp_min(1e-30)).max().item()
        r7 = ((dv.sum(0) - g.sum(0)).abs() / dv.abs().sum(0).clamp_min(1e-30)).max().item()
        a8 = (q * dq).sum(dim=(0, 2))
        b8 = (k * dk).sum(dim=(0, 2))
        r8 = ((a8 - b8).abs() / ((q * dq).abs().sum(dim=(0, 2)) + (k * dk).abs().sum(dim=(0, 2)))).max().item()
        worst["sum_dk"] = max(worst["sum_dk"], r6)
        worst["sum_dv"] = max(worst["sum_dv"], r7)
        worst["qdq_kdk"] = max(worst["qdq_kdk"], r8)
    log(f"{name}: invariant residuals {worst}")
    # bf16 rounding leaves residuals of ~1e-3 of the summed magnitudes (measured <= 6e-4 for the
    # sums and <= 2e-5 for the inner products on all four workloads).
    assert worst["sum_dk"] <= 5e-3 and worst["sum_dv"] <= 5e-3, worst
    assert worst["qdq_kdk"] <= 1e-3, worst


@pytest.mark.timeout(600)
def test_full_size_uniform():
    check_full_oracle("uniform")
    check_invariants("uniform")


@pytest.mark.timeout(600)
def test_full_size_hetero():
    pack, _ = workload_run("hetero")
    check_full_oracle("hetero", heads=[0, pack.heads // 2, pack.heads - 1])
    check_query_rows("hetero")
    check_invariants("hetero")
    check_key_rows("hetero", seq=int(np.argmax(np.diff(pack.cu_seqlens))), head=5, nkeys=None)


@pytest.mark.timeout(900)
def test_full_size_long():
    check_query_rows("long")
    check_invariants("long")
    pack, _ = workload_run("long")
    check_key_rows("long", seq=0, head=pack.heads // 2, nkeys=None, torch_backend=True)


@pytest.mark.timeout(900)
def test_full_size_skew():
    check_query_rows("skew")
    check_invariants("skew")
    check_short_clips("skew", 1024, max_clips=2)
    pack, _ = workload_run("skew")
    check_key_rows("skew", seq=int(np.argmax(np.diff(pack.cu_seqlens))), head=pack.heads // 2, nkeys=None,
                   torch_backend=True)
