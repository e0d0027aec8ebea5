"""Pins for the float64 oracle, checked against facts that do not come from it.

Each pin comes from the mathematics of softmax attention (the paper prints no
attention values): closed forms for degenerate clips, invariants of the
softmax Jacobian, finite differences, an independent library routine (torch's
scaled_dot_product_attention with autograd, float64 on the CPU) and a
pure-Python brute force. ``test_mutants_are_caught`` plants one plausible
mistake at a time in a copy of the oracle and checks that some pin fails.
"""
import math
import types

import numpy as np
import pytest

import oracle.varlen_attention as orc
from paper_2607_01701_amd.workload import cu_from_lengths, make_pack


def rand_pack(lengths, H, D, seed, dtype=np.float64):
    rng = np.random.default_rng(seed)
    T = int(sum(lengths))
    cu = cu_from_lengths(lengths)
    q, k, v, do = (rng.standard_normal((T, H, D)).astype(dtype) for _ in range(4))
    return cu, q, k, v, do


def rel(a, b):
    den = max(float(np.max(np.abs(b))), 1e-300)
    return float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) / den


# ---------------------------------------------------------------- closed forms

def check_len1(mod):
    """P1: a one-token clip attends only to itself."""
    cu, q, k, v, do = rand_pack([1, 1], 2, 8, 1)
    sc = 0.37
    r = mod.attention(q, k, v, do, cu, sc)
    ok = np.allclose(r["out"], v, rtol=0, atol=1e-15)
    ok &= np.allclose(r["lse"].T, sc * np.sum(q * k, axis=2), rtol=0, atol=1e-14)
    ok &= np.all(np.abs(r["dq"]) < 1e-15) and np.all(np.abs(r["dk"]) < 1e-15)
    ok &= np.allclose(r["dv"], do, rtol=0, atol=1e-15)
    return bool(ok)


def check_equal_v(mod):
    """P2: identical value rows give that row as output."""
    cu, q, k, v, do = rand_pack([9, 4], 2, 8, 2)
    for s in range(2):
        a, b = cu[s], cu[s + 1]
        v[a:b] = v[a]
    r = mod.attention(q, k, v, do, cu, 0.5)
    return bool(np.allclose(r["out"][:9], np.broadcast_to(v[0], (9, 2, 8)), atol=1e-13)
                and np.allclose(r["out"][9:], np.broadcast_to(v[9], (4, 2, 8)), atol=1e-13))


def check_equal_k(mod):
    """P3: identical key rows give uniform weights: mean of V, lse = s*q.k + ln L, dq = 0."""
    L = 11
    cu, q, k, v, do = rand_pack([L], 2, 8, 3)
    k[:] = k[0]
    sc = 0.3
    r = mod.attention(q, k, v, do, cu, sc)
    ok = np.allclose(r["out"], np.broadcast_to(v.mean(axis=0), v.shape), atol=1e-13)
    lse_ref = sc * np.einsum("thd,hd->ht", q, k[0]) + math.log(L)
    ok &= np.allclose(r["lse"], lse_ref, atol=1e-13)
    ok &= np.all(np.abs(r["dq"]) < 1e-12)
    return bool(ok)


def check_len2_by_hand(mod):
    """P4: two tokens, D = 1: p = sigmoid(s00 - s01), all gradients in closed form."""
    qv, kv, vv, dov = [0.7, -1.3], [0.4, 1.1], [2.0, -0.5], [0.3, 1.7]
    sc = 0.9
    q = np.array(qv).reshape(2, 1, 1)
    k = np.array(kv).reshape(2, 1, 1)
    v = np.array(vv).reshape(2, 1, 1)
    do = np.array(dov).reshape(2, 1, 1)
    r = mod.attention(q, k, v, do, np.array([0, 2]), sc)
    ok = True
    for i in range(2):
        s0, s1 = sc * qv[i] * kv[0], sc * qv[i] * kv[1]
        p0 = 1.0 / (1.0 + math.exp(-(s0 - s1)))
        p1 = 1.0 - p0
        o = p0 * vv[0] + p1 * vv[1]
        lse = max(s0, s1) + math.log(math.exp(s0 - max(s0, s1)) + math.exp(s1 - max(s0, s1)))
        # d<do, o>/dq_i = do_i * sc * p0 p1 (k0 - k1)(v0 - v1)
        dq = dov[i] * sc * p0 * p1 * (kv[0] - kv[1]) * (vv[0] - vv[1])
        ok &= abs(r["out"][i, 0, 0] - o) < 1e-14
        ok &= abs(r["lse"][0, i] - lse) < 1e-14
        ok &= abs(r["dq"][i, 0, 0] - dq) < 1e-14
    # dv_j = sum_i p_ij do_i ; dk_j = sum_i sc q_i p_ij (do_i (v_j - o_i))
    dv = [0.0, 0.0]
    dk = [0.0, 0.0]
    for i in range(2):
        s = [sc * qv[i] * kv[0], sc * qv[i] * kv[1]]
        p = [1.0 / (1.0 + math.exp(s[1] - s[0]))]
        p.append(1.0 - p[0])
        o = p[0] * vv[0] + p[1] * vv[1]
        for j in range(2):
            dv[j] += p[j] * dov[i]
            dk[j] += sc * qv[i] * p[j] * dov[i] * (vv[j] - o)
    for j in range(2):
        ok &= abs(r["dv"][j, 0, 0] - dv[j]) < 1e-14
        ok &= abs(r["dk"][j, 0, 0] - dk[j]) < 1e-14
    return bool(ok)


# ---------------------------------------------------------------- invariants

def check_invariants(mod):
    """P6 sum dk = 0; P7 sum dv = sum dout; P8 <Q,dQ> = <K,dK>, per clip and head."""
    lens = [5, 17, 1, 30]
    cu, q, k, v, do = rand_pack(lens, 3, 8, 4)
    r = mod.attention(q, k, v, do, cu, 0.35)
    ok = True
    for s in range(len(lens)):
        a, b = cu[s], cu[s + 1]
        for h in range(3):
            dk, dv, dq = r["dk"][a:b, h], r["dv"][a:b, h], r["dq"][a:b, h]
            ok &= np.max(np.abs(dk.sum(0))) < 1e-12
            ok &= np.allclose(dv.sum(0), do[a:b, h].sum(0), atol=1e-12)
            ok &= abs(np.sum(q[a:b, h] * dq) - np.sum(k[a:b, h] * dk)) < 1e-11
    return bool(ok)


def check_delta_identity(mod):
    """P9: Delta_i = sum_j P_ij dP_ij, with P and dP from plain loops."""
    L, D, sc = 6, 4, 0.6
    cu, q, k, v, do = rand_pack([L], 1, D, 5)
    r = mod.attention(q, k, v, do, cu, sc)
    ok = True
    for i in range(L):
        s = [sc * sum(q[i, 0, d] * k[j, 0, d] for d in range(D)) for j in range(L)]
        m = max(s)
        e = [math.exp(x - m) for x in s]
        z = sum(e)
        tot = sum(e[j] / z * sum(do[i, 0, d] * v[j, 0, d] for d in range(D)) for j in range(L))
        ok &= abs(r["delta"][0, i] - tot) < 1e-13
    return bool(ok)


def check_key_shift(mod):
    """P10: adding c to every key leaves out unchanged and adds scale*q.c to lse."""
    cu, q, k, v, do = rand_pack([7, 12], 2, 8, 6)
    c = np.random.default_rng(60).standard_normal(8)
    sc = 0.4
    r0 = mod.attention(q, k, v, do, cu, sc)
    r1 = mod.attention(q, k + c, v, do, cu, sc)
    ok = np.allclose(r0["out"], r1["out"], atol=1e-12)
    ok &= np.allclose(r1["lse"] - r0["lse"], sc * np.einsum("thd,d->ht", q, c), atol=1e-12)
    return bool(ok)


def check_permutation_isolation(mod):
    """P11: permuting clips permutes every output; editing one clip leaves the others."""
    lens = [4, 9, 2, 13]
    cu, q, k, v, do = rand_pack(lens, 2, 4, 7)
    sc = 0.5
    r = mod.attention(q, k, v, do, cu, sc)
    perm = [2, 0, 3, 1]
    idx = np.concatenate([np.arange(cu[s], cu[s + 1]) for s in perm])
    cu2 = cu_from_lengths([lens[s] for s in perm])
    r2 = mod.attention(q[idx], k[idx], v[idx], do[idx], cu2, sc)
    ok = True
    for key in ("out", "dq", "dk", "dv"):
        ok &= np.allclose(r2[key], r[key][idx], atol=1e-13)
    for key in ("lse", "delta"):
        ok &= np.allclose(r2[key], r[key][:, idx], atol=1e-13)
    q3 = q.copy()
    q3[cu[1]:cu[2]] += 1.0  # edit clip 1 only
    r3 = mod.attention(q3, k, v, do, cu, sc)
    others = np.r_[cu[0]:cu[1], cu[2]:cu[4]]
    for key in ("out", "dq", "dk", "dv"):
        ok &= np.array_equal(r3[key][others], r[key][others])
    return bool(ok)


# ---------------------------------------------------------------- gradients

def check_finite_differences(mod, lens=(1, 2, 3, 5, 17), H=2, D=4, seed=8):
    """P12: dq, dk, dv equal central differences of <dout, out> (h = 1e-6)."""
    cu, q, k, v, do = rand_pack(list(lens), H, D, seed)
    sc = 0.45
    r = mod.attention(q, k, v, do, cu, sc)

    def f(qq, kk, vv):
        return float(np.sum(do * mod.attention(qq, kk, vv, do, cu, sc)["out"]))

    h = 1e-6
    ok = True
    for name, arr, pos in (("dq", q, 0), ("dk", k, 1), ("dv", v, 2)):
        g = np.zeros_like(arr)
        for ix in np.ndindex(arr.shape):
            args_p = [q, k, v]
            args_m = [q, k, v]
            xp = arr.copy()
            xm = arr.copy()
            xp[ix] += h
            xm[ix] -= h
            args_p[pos] = xp
            args_m[pos] = xm
            g[ix] = (f(*args_p) - f(*args_m)) / (2 * h)
        ok &= rel(r[name], g) < 1e-6
    return bool(ok)


def torch_reference(cu, q, k, v, do, sc):
    """torch's SDPA (math path, float64, CPU) with a block-diagonal mask + autograd."""
    import torch
    T, H, D = q.shape
    seg = np.zeros(T, dtype=np.int64)
    for s in range(len(cu) - 1):
        seg[cu[s]:cu[s + 1]] = s
    segt = torch.from_numpy(seg)
    mask = segt[:, None] == segt[None, :]
    tq, tk, tv = (torch.tensor(np.ascontiguousarray(x.transpose(1, 0, 2))[None], dtype=torch.float64,
                               requires_grad=True) for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=sc)
    tdo = torch.tensor(np.ascontiguousarray(do.transpose(1, 0, 2))[None], dtype=torch.float64)
    out.backward(tdo)
    scores = sc * (tq.detach() @ tk.detach().transpose(-1, -2))
    scores = scores.masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(scores, dim=-1)[0]

    def back(t):
        return t[0].detach().numpy().transpose(1, 0, 2)

    return {"out": back(out), "dq": back(tq.grad), "dk": back(tk.grad), "dv": back(tv.grad),
            "lse": lse.numpy()}


def check_torch_sdpa(mod):
    """P15: agrees with torch's scaled_dot_product_attention + autograd to 1e-10."""
    lens = [3, 1, 16, 7, 33]
    cu, q, k, v, do = rand_pack(lens, 2, 8, 9)
    sc = 1 / math.sqrt(8)
    r = mod.attention(q, k, v, do, cu, sc)
    t = torch_reference(cu, q, k, v, do, sc)
    ok = True
    for key in ("out", "dq", "dk", "dv", "lse"):
        ok &= rel(r[key], t[key]) < 1e-10
    return bool(ok)


def brute_force(cu, q, k, v, do, sc):
    """Pure-Python loops (no BLAS, math.exp) over the same definition."""
    T, H, D = q.shape
    res = {n: np.zeros((T, H, D)) for n in ("out", "dq", "dk", "dv")}
    res["lse"] = np.zeros((H, T))
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        L = b - a
        for h in range(H):
            Q = [[float(q[a + i, h, d]) for d in range(D)] for i in range(L)]
            K = [[float(k[a + i, h, d]) for d in range(D)] for i in range(L)]
            V = [[float(v[a + i, h, d]) for d in range(D)] for i in range(L)]
            G = [[float(do[a + i, h, d]) for d in range(D)] for i in range(L)]
            P = []
            for i in range(L):
                srow = [sc * sum(Q[i][d] * K[j][d] for d in range(D)) for j in range(L)]
                m = max(srow)
                e = [math.exp(x - m) for x in srow]
                z = math.fsum(e)
                P.append([x / z for x in e])
                res["lse"][h, a + i] = m + math.log(z)
            O = [[math.fsum(P[i][j] * V[j][d] for j in range(L)) for d in range(D)] for i in range(L)]
            for i in range(L):
                dl = math.fsum(G[i][d] * O[i][d] for d in range(D))
                for j in range(L):
                    dp = math.fsum(G[i][d] * V[j][d] for d in range(D))
                    ds = P[i][j] * (dp - dl)
                    for d in range(D):
                        res["dq"][a + i, h, d] += sc * ds * K[j][d]
                        res["dk"][a + j, h, d] += sc * ds * Q[i][d]
                        res["dv"][a + j, h, d] += P[i][j] * G[i][d]
                for d in range(D):
                    res["out"][a + i, h, d] = O[i][d]
    return res


def check_brute_force(mod):
    """P13: the blocked BLAS oracle equals plain loops to 1e-12."""
    lens = [1, 2, 3, 5, 17]
    cu, q, k, v, do = rand_pack(lens, 2, 4, 10)
    r = mod.attention(q, k, v, do, cu, 0.55)
    b = brute_force(cu, q, k, v, do, 0.55)
    return all(rel(r[key], b[key]) < 1e-12 for key in ("out", "dq", "dk", "dv", "lse"))


def check_dominant_key(mod):
    """P16: one key's score exceeds every other by 1,000 (natural units): the softmax is
    exactly one-hot in float64, so out = that key's value row, lse = its score, dq = dk = 0
    (up to rounding), and dv is the summed dout on that key, zero elsewhere. Scores this large also overflow
    any exponential taken without subtracting the row maximum."""
    L, D, star = 6, 8, 3
    cu, q, k, v, do = rand_pack([L], 1, D, 16)
    q[:, 0, :] = 0.0
    q[:, 0, 0] = 50.0
    k[:, 0, 0] = 0.0  # other dimensions keep their noise, orthogonal to every query
    k[star, 0, 0] = 40.0
    sc = 0.5  # scores: 1,000 on the dominant key, exactly 0 elsewhere
    r = mod.attention(q, k, v, do, cu, sc)
    ok = np.array_equal(r["out"][:, 0], np.broadcast_to(v[star, 0], (L, D)))
    ok &= np.array_equal(r["lse"][0], np.full(L, 1000.0))
    # dS = P (dP - Delta) vanishes: on the dominant key dP and Delta are the same dot product
    # (rounded along two summation paths), elsewhere P = 0.
    ok &= np.all(np.abs(r["dq"]) < 1e-12) and np.all(np.abs(r["dk"]) < 1e-12)
    dv = np.zeros((L, D))
    dv[star] = do[:, 0].sum(axis=0)
    ok &= np.allclose(r["dv"][:, 0], dv, rtol=0, atol=1e-13)
    return bool(ok)


PINS = {
    "P16_dominant_key": check_dominant_key,
    "P1_len1": check_len1,
    "P2_equal_v": check_equal_v,
    "P3_equal_k": check_equal_k,
    "P4_len2_by_hand": check_len2_by_hand,
    "P6_P7_P8_invariants": check_invariants,
    "P9_delta": check_delta_identity,
    "P10_key_shift": check_key_shift,
    "P11_permutation_isolation": check_permutation_isolation,
    "P12_finite_differences": check_finite_differences,
    "P13_brute_force": check_brute_force,
    "P15_torch_sdpa": check_torch_sdpa,
}


@pytest.mark.parametrize("name", sorted(PINS))
def test_pin(name):
    assert PINS[name](orc), name


def test_rows_sum_to_one():
    """P5: the oracle's own row check (|sum_j P_ij - 1| <= 1e-12) holds."""
    cu, q, k, v, do = rand_pack([40, 3, 100], 2, 16, 11)
    orc.attention(q, k, v, do, cu, 1.7, check_rows=True)


@pytest.mark.parametrize("block", [1, 7, 100, 512])
def test_block_size_independence(block):
    """P14: the row-block size changes nothing beyond rounding."""
    cu, q, k, v, do = rand_pack([100, 37], 2, 8, 12)
    ref = orc.attention(q, k, v, do, cu, 0.3, block_rows=100)
    r = orc.attention(q, k, v, do, cu, 0.3, block_rows=block)
    for key in ("out", "dq", "dk", "dv", "lse", "delta"):
        assert rel(r[key], ref[key]) < 1e-12, key


def test_heads_independent():
    """P11 (heads): computing a head subset gives the same values for those heads."""
    cu, q, k, v, do = rand_pack([20, 9], 4, 8, 13)
    full = orc.attention(q, k, v, do, cu, 0.4)
    sub = orc.attention(q, k, v, do, cu, 0.4, heads=[1, 3])
    for key in ("out", "dq", "dk", "dv"):
        assert np.array_equal(sub[key][:, [1, 3]], full[key][:, [1, 3]])
        assert np.all(sub[key][:, [0, 2]] == 0)


def test_zero_length_clips_skipped():
    """Empty clips contribute nothing and disturb nothing."""
    cu, q, k, v, do = rand_pack([5, 0, 6, 0], 2, 4, 14)
    r = orc.attention(q, k, v, do, cu, 0.5)
    cu2 = cu_from_lengths([5, 6])
    r2 = orc.attention(q, k, v, do, cu2, 0.5)
    for key in ("out", "dq", "dk", "dv", "lse"):
        assert np.array_equal(r[key], r2[key])


def test_query_rows_match_full():
    """Row-sampled out/lse/dq equal the full oracle at those rows."""
    lens = [50, 1, 70]
    cu, q, k, v, do = rand_pack(lens, 3, 8, 15)
    full = orc.attention(q, k, v, do, cu, 0.3)
    toks = [0, 49, 50, 51, 120, 77]
    hs = [0, 2, 1, 0, 2, 1]
    r = orc.query_rows(q, k, v, do, cu, 0.3, toks, hs)
    for i, (t, h) in enumerate(zip(toks, hs)):
        assert np.allclose(r["out"][i], full["out"][t, h], atol=1e-13)
        assert abs(r["lse"][i] - full["lse"][h, t]) < 1e-13
        assert np.allclose(r["dq"][i], full["dq"][t, h], atol=1e-13)


def test_key_rows_match_full():
    """Key-sampled dk/dv equal the full oracle at those keys."""
    lens = [30, 90]
    cu, q, k, v, do = rand_pack(lens, 2, 8, 16)
    full = orc.attention(q, k, v, do, cu, 0.3)
    keys = [0, 5, 89]
    r = orc.key_rows(q, k, v, do, cu, 0.3, seq=1, head=1, keys=keys, block_rows=17)
    for i, j in enumerate(keys):
        assert np.allclose(r["dk"][i], full["dk"][30 + j, 1], atol=1e-13)
        assert np.allclose(r["dv"][i], full["dv"][30 + j, 1], atol=1e-13)


def test_bf16_inputs_are_exact():
    """The oracle sees the generator's bf16 values exactly (float32 widening is lossless)."""
    p = make_pack([33, 5], 2, 8, seed=3)
    q = p.f32("q")
    assert q.dtype == np.float32
    assert np.array_equal(q.astype(np.float64).astype(np.float32), q)
    # bf16 values have only 8 significant bits: the low 16 bits of float32 are zero
    assert np.all((q.view(np.uint32) & 0xFFFF) == 0)


# ---------------------------------------------------------------- planted mistakes

MUTANTS = {
    "softmax_unnormalised": ("return E / l[:, None], m, l", "return E, m, l"),
    "dS_sign": ("P * (dP - delta[:, None])", "P * (dP + delta[:, None])"),
    "dK_no_scale": ("dK += scale * (dS.T @ Qb)", "dK += (dS.T @ Qb)"),
    "dV_transposed": ("dV += P.T @ dOb", "dV += P @ dOb"),
    "lse_log2": ("lse[r0:r1] = m + np.log(l)", "lse[r0:r1] = m + np.log2(l)"),
    "lse_no_max": ("lse[r0:r1] = m + np.log(l)", "lse[r0:r1] = np.log(l)"),
    "delta_from_v": ("db = np.sum(dOb * Ob, axis=1)", "db = np.sum(dOb * V[r0:r1], axis=1)"),
    "scores_no_scale": ("return scale * (Qb @ K.T)", "return (Qb @ K.T)"),
    "dQ_uses_V": ("dQ[r0:r1] = scale * (dS @ K)", "dQ[r0:r1] = scale * (dS @ V)"),
    "dK_uses_K": ("dK += scale * (dS.T @ Qb)", "dK += scale * (dS.T @ K[r0:r1])"),
    "dP_uses_K": ("dP = dOb @ V.T", "dP = dOb @ K.T"),
    "softmax_no_max_shift": ("E = np.exp(S - m[:, None])", "E = np.exp(S)"),
}


def mutant_module(old, new):
    src = open(orc.__file__).read()
    assert src.count(old) >= 1, f"mutation site not found: {old}"
    mod = types.ModuleType("oracle_mutant")
    exec(compile(src.replace(old, new), "oracle_mutant", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutants_are_caught(name):
    mod = mutant_module(*MUTANTS[name])
    failing = []
    for pin, fn in PINS.items():
        if pin in ("P12_finite_differences", "P13_brute_force"):
            continue  # the cheaper pins must already catch every mutant
        try:
            with np.errstate(over="ignore", invalid="ignore", divide="ignore"):  # mutants may overflow
                if not fn(mod):
                    failing.append(pin)
        except Exception:  # a shape error is also a detection
            failing.append(pin)
    assert failing, f"mutant {name} passed every pin"


def test_key_rows_torch_matches_full():
    """The torch variant of the key-column routine equals the full oracle at those keys."""
    lens = [30, 90]
    cu, q, k, v, do = rand_pack(lens, 2, 8, 17)
    full = orc.attention(q, k, v, do, cu, 0.3)
    keys = [0, 44, 89]
    r = orc.key_rows_torch(q, k, v, do, cu, 0.3, seq=1, head=0, keys=keys, block_rows=13)
    for i, j in enumerate(keys):
        assert np.allclose(r["dk"][i], full["dk"][30 + j, 0], atol=1e-13)
        assert np.allclose(r["dv"][i], full["dv"][30 + j, 0], atol=1e-13)


# ---------------------------------------------------------------- cross-attention pins
#
# Queries of sequence s at rows cu_q[s] .. cu_q[s+1], keys/values at cu_k[s] .. cu_k[s+1]
# (Wan2.1's cross-attention, Section V-A; text conditioning, Section II-A; text under 256
# tokens, Section IV-B footnote). Each pin below is fixed by the mathematics, as above.

def rand_cross(lq, lk, H, D, seed):
    rng = np.random.default_rng(seed)
    cuq, cuk = cu_from_lengths(lq), cu_from_lengths(lk)
    q, do = (rng.standard_normal((int(cuq[-1]), H, D)) for _ in range(2))
    k, v = (rng.standard_normal((int(cuk[-1]), H, D)) for _ in range(2))
    return cuq, cuk, q, k, v, do


def check_cross_one_key(mod):
    """X1: one key per sequence: out = v0 for every query, lse = s q.k0, dq = dk = 0, dv0 = sum dO."""
    cuq, cuk, q, k, v, do = rand_cross([5, 3], [1, 1], 2, 8, 21)
    sc = 0.41
    r = mod.attention(q, k, v, do, cuq, sc, cu_seqlens_k=cuk)
    ok = True
    for s in range(2):
        a, b, j = cuq[s], cuq[s + 1], cuk[s]
        ok &= np.allclose(r["out"][a:b], np.broadcast_to(v[j], (b - a,) + v.shape[1:]), atol=1e-14)
        ok &= np.allclose(r["lse"][:, a:b].T, sc * np.einsum("thd,hd->th", q[a:b], k[j]), atol=1e-13)
        ok &= np.allclose(r["dv"][j], do[a:b].sum(axis=0), atol=1e-13)
    ok &= np.all(np.abs(r["dq"]) < 1e-14) and np.all(np.abs(r["dk"]) < 1e-13)
    return bool(ok)


def check_cross_equal_keys(mod):
    """X2: identical keys: uniform weights over the Lk keys: mean of V, lse = s q.k + ln Lk, dq = 0."""
    cuq, cuk, q, k, v, do = rand_cross([7], [13], 2, 8, 22)
    k[:] = k[0]
    sc = 0.3
    r = mod.attention(q, k, v, do, cuq, sc, cu_seqlens_k=cuk)
    ok = np.allclose(r["out"], np.broadcast_to(v.mean(axis=0), q.shape), atol=1e-13)
    ok &= np.allclose(r["lse"], sc * np.einsum("thd,hd->ht", q, k[0]) + math.log(13), atol=1e-13)
    ok &= np.all(np.abs(r["dq"]) < 1e-12)
    return bool(ok)


def check_cross_invariants(mod):
    """X3: per (sequence, head): sum_j dk_j = 0, sum_j dv_j = sum_i dO_i, <Q, dQ> = <K, dK>."""
    lq, lk = [5, 17, 1, 30], [9, 2, 4, 1]
    cuq, cuk, q, k, v, do = rand_cross(lq, lk, 3, 8, 23)
    r = mod.attention(q, k, v, do, cuq, 0.35, cu_seqlens_k=cuk)
    ok = True
    for s in range(len(lq)):
        a, b, ka, kb = cuq[s], cuq[s + 1], cuk[s], cuk[s + 1]
        for h in range(3):
            dk, dv, dq = r["dk"][ka:kb, h], r["dv"][ka:kb, h], r["dq"][a:b, h]
            ok &= np.max(np.abs(dk.sum(0))) < 1e-12
            ok &= np.allclose(dv.sum(0), do[a:b, h].sum(0), atol=1e-12)
            ok &= abs(np.sum(q[a:b, h] * dq) - np.sum(k[ka:kb, h] * dk)) < 1e-11
    return bool(ok)


def torch_reference_cross(cuq, cuk, q, k, v, do, sc):
    """torch SDPA (math path, float64, CPU) with a rectangular block mask + autograd."""
    import torch
    segq = np.repeat(np.arange(len(cuq) - 1), np.diff(cuq))
    segk = np.repeat(np.arange(len(cuk) - 1), np.diff(cuk))
    mask = torch.from_numpy(segq)[:, None] == torch.from_numpy(segk)[None, :]
    tq, tk, tv = (torch.tensor(np.ascontiguousarray(x.transpose(1, 0, 2))[None], dtype=torch.float64,
                               requires_grad=True) for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask, scale=sc)
    out.backward(torch.tensor(np.ascontiguousarray(do.transpose(1, 0, 2))[None], dtype=torch.float64))
    scores = (sc * (tq.detach() @ tk.detach().transpose(-1, -2))).masked_fill(~mask, float("-inf"))
    lse = torch.logsumexp(scores, dim=-1)[0]

    def back(t):
        return t[0].detach().numpy().transpose(1, 0, 2)

    return {"out": back(out), "dq": back(tq.grad), "dk": back(tk.grad), "dv": back(tv.grad), "lse": lse.numpy()}


def check_cross_torch_sdpa(mod):
    """X4: agrees with torch's scaled_dot_product_attention + autograd (rectangular mask) to 1e-10."""
    lq, lk = [3, 1, 16, 7, 33], [5, 4, 1, 20, 9]
    cuq, cuk, q, k, v, do = rand_cross(lq, lk, 2, 8, 24)
    sc = 1 / math.sqrt(8)
    r = mod.attention(q, k, v, do, cuq, sc, cu_seqlens_k=cuk)
    t = torch_reference_cross(cuq, cuk, q, k, v, do, sc)
    return all(rel(r[key], t[key]) < 1e-10 for key in ("out", "dq", "dk", "dv", "lse"))


def check_cross_finite_differences(mod):
    """X5: dq, dk, dv of a cross pack equal central differences of <dout, out> (h = 1e-6)."""
    cuq, cuk, q, k, v, do = rand_cross([3, 1, 4], [2, 5, 1], 2, 4, 25)
    sc = 0.45
    r = mod.attention(q, k, v, do, cuq, sc, cu_seqlens_k=cuk)

    def f(qq, kk, vv):
        return float(np.sum(do * mod.attention(qq, kk, vv, do, cuq, sc, cu_seqlens_k=cuk)["out"]))

    h = 1e-6
    ok = True
    for name, arr, pos in (("dq", q, 0), ("dk", k, 1), ("dv", v, 2)):
        g = np.zeros_like(arr)
        for ix in np.ndindex(arr.shape):
            xp, xm = arr.copy(), arr.copy()
            xp[ix] += h
            xm[ix] -= h
            ap, am = [q, k, v], [q, k, v]
            ap[pos], am[pos] = xp, xm
            g[ix] = (f(*ap) - f(*am)) / (2 * h)
        ok &= rel(r[name], g) < 1e-6
    return bool(ok)


def brute_force_cross(cuq, cuk, q, k, v, do, sc):
    """Pure-Python loops over the cross-attention definition (no BLAS)."""
    Tq, H, D = q.shape
    res = {n: np.zeros((Tq, H, D)) for n in ("out", "dq")}
    res.update({n: np.zeros((k.shape[0], H, D)) for n in ("dk", "dv")})
    res["lse"] = np.zeros((H, Tq))
    for s in range(len(cuq) - 1):
        a, b, ka, kb = int(cuq[s]), int(cuq[s + 1]), int(cuk[s]), int(cuk[s + 1])
        for h in range(H):
            for i in range(a, b):
                srow = [sc * math.fsum(q[i, h, d] * k[j, h, d] for d in range(D)) for j in range(ka, kb)]
                m = max(srow)
                e = [math.exp(x - m) for x in srow]
                z = math.fsum(e)
                p = [x / z for x in e]
                res["lse"][h, i] = m + math.log(z)
                o = [math.fsum(p[j] * v[ka + j, h, d] for j in range(kb - ka)) for d in range(D)]
                res["out"][i, h] = o
                dl = math.fsum(do[i, h, d] * o[d] for d in range(D))
                for j in range(kb - ka):
                    dp = math.fsum(do[i, h, d] * v[ka + j, h, d] for d in range(D))
                    ds = p[j] * (dp - dl)
                    for d in range(D):
                        res["dq"][i, h, d] += sc * ds * k[ka + j, h, d]
                        res["dk"][ka + j, h, d] += sc * ds * q[i, h, d]
                        res["dv"][ka + j, h, d] += p[j] * do[i, h, d]
    return res


def check_cross_brute_force(mod):
    """X6: the blocked BLAS oracle equals plain loops on a cross pack to 1e-12."""
    cuq, cuk, q, k, v, do = rand_cross([1, 6, 3], [4, 1, 7], 2, 4, 26)
    r = mod.attention(q, k, v, do, cuq, 0.55, cu_seqlens_k=cuk)
    b = brute_force_cross(cuq, cuk, q, k, v, do, 0.55)
    return all(rel(r[key], b[key]) < 1e-12 for key in ("out", "dq", "dk", "dv", "lse"))


CROSS_PINS = {
    "X1_one_key": check_cross_one_key,
    "X2_equal_keys": check_cross_equal_keys,
    "X3_invariants": check_cross_invariants,
    "X4_torch_sdpa": check_cross_torch_sdpa,
    "X5_finite_differences": check_cross_finite_differences,
    "X6_brute_force": check_cross_brute_force,
}


@pytest.mark.parametrize("name", sorted(CROSS_PINS))
def test_cross_pin(name):
    assert CROSS_PINS[name](orc), name


def test_cross_self_case_is_self_attention():
    """cu_seqlens_k = cu_seqlens reproduces the self-attention results exactly."""
    cu, q, k, v, do = rand_pack([9, 4, 1], 2, 8, 27)
    a = orc.attention(q, k, v, do, cu, 0.4)
    b = orc.attention(q, k, v, do, cu, 0.4, cu_seqlens_k=cu)
    for key in ("out", "dq", "dk", "dv", "lse", "delta"):
        assert np.array_equal(a[key], b[key])


def test_cross_rejects_queries_without_keys():
    cuq, cuk, q, k, v, do = rand_cross([3, 2], [4, 1], 1, 4, 28)
    with pytest.raises(ValueError):
        orc.attention(q, k[:4], v[:4], do, cuq, 0.5, cu_seqlens_k=np.array([0, 4, 4]))


def test_cross_query_and_key_rows_match_full():
    """The row- and column-sampled routines follow the key offsets too."""
    cuq, cuk, q, k, v, do = rand_cross([40, 25], [7, 30], 2, 8, 29)
    full = orc.attention(q, k, v, do, cuq, 0.3, cu_seqlens_k=cuk)
    toks, hs = [0, 39, 40, 64], [1, 0, 1, 0]
    r = orc.query_rows(q, k, v, do, cuq, 0.3, toks, hs, cu_seqlens_k=cuk)
    for i, (t, h) in enumerate(zip(toks, hs)):
        assert np.allclose(r["out"][i], full["out"][t, h], atol=1e-13)
        assert abs(r["lse"][i] - full["lse"][h, t]) < 1e-13
        assert np.allclose(r["dq"][i], full["dq"][t, h], atol=1e-13)
    keys = [0, 13, 29]
    for fn in (orc.key_rows, orc.key_rows_torch):
        r = fn(q, k, v, do, cuq, 0.3, seq=1, head=1, keys=keys, block_rows=11, cu_seqlens_k=cuk)
        for i, j in enumerate(keys):
            assert np.allclose(r["dk"][i], full["dk"][7 + j, 1], atol=1e-13)
            assert np.allclose(r["dv"][i], full["dv"][7 + j, 1], atol=1e-13)


CROSS_MUTANTS = {
    "keys_at_query_offsets": ("q[a:b, h], k[ka:kb, h], v[ka:kb, h], dout[a:b, h]",
                              "q[a:b, h], k[a:b, h], v[a:b, h], dout[a:b, h]"),
    "dk_written_at_query_rows": ('res["dk"][ka:kb, h] = dK', 'res["dk"][a:b, h] = dK[: b - a]'),
    "dv_written_at_query_rows": ('res["dv"][ka:kb, h] = dV', 'res["dv"][a:b, h] = dV[: b - a]'),
}


@pytest.mark.parametrize("name", sorted(CROSS_MUTANTS) + sorted(MUTANTS))
def test_cross_mutants_are_caught(name):
    """Plausible mistakes in the cross-attention plumbing (and the arithmetic mutants above)
    fail at least one cheap cross pin."""
    mod = mutant_module(*(CROSS_MUTANTS.get(name) or MUTANTS[name]))
    failing = []
    for pin, fn in CROSS_PINS.items():
        if pin in ("X5_finite_differences", "X6_brute_force"):
            continue
        try:
            if not fn(mod):
                failing.append(pin)
        except Exception:
            failing.append(pin)
    assert failing, f"mutant {name} passed every cross pin"
