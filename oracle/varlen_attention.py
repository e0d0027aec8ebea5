"""Float64 CPU oracle for packed variable-length bidirectional attention.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or run
this module; only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it. It shares no code with the HIP
path and imports nothing from the package.

What it computes (Section III, Observation 2: full self-attention over the
unified token sequence of one clip, whose cost grows as O(L^2); Eq. (9) carries
the same term as alpha_2 * B * S^2; the backward pass of the DiT appears in the
Fig. 1 caption). The paper gives no formulas for the operator itself, so the
oracle is the plain definition of scaled dot-product attention and its exact
gradient, for each clip s (rows cu[s] .. cu[s+1]) and each head h independently:

    S   = scale * Q K^T
    P   = row-softmax(S)                 (full row: every key of the clip)
    O   = P V
    LSE = m + ln(sum_j exp(S_ij - m)),   m = max_j S_ij   (natural log)
    Delta_i = sum_d dO_id O_id
    dV  = P^T dO
    dP  = dO V^T
    dS  = P * (dP - Delta)
    dQ  = scale * dS K
    dK  = scale * dS^T Q

Gradients are those of the scalar <dout, out>; LSE is an output only.
There is no causal mask: attention is block-diagonal over the clips.

Cross-attention (queries and keys from different token streams): Wan2.1, one of
the paper's models, uses self- and cross-attention (Section V-A), and the DiT is
conditioned on text (Section II-A) whose sequences are short, typically under
256 tokens (Section IV-B footnote). Reading: sequence s then has its queries at
rows cu_q[s] .. cu_q[s+1] of q / dout and its keys and values at rows
cu_k[s] .. cu_k[s+1] of k / v; every formula above holds with Q [Lq, D] and
K, V [Lk, D], the softmax running over the Lk keys. A sequence with queries but
no keys has no defined softmax and is rejected. Without cu_k, cu_k = cu_q.

Every floating-point step runs in float64 on the bf16 inputs widened exactly.
Rows are processed in blocks; each block forms its complete score rows over
all L keys, so no running-max rescaling is ever needed.

Parity status of each function is pinned by ``tests/test_oracle.py``.
"""
from __future__ import annotations

import numpy as np

LN2 = float(np.log(2.0))


def _scores(Qb: np.ndarray, K: np.ndarray, scale: float) -> np.ndarray:
    """S = scale * Q K^T for one row block."""
    return scale * (Qb @ K.T)


def _row_softmax(S: np.ndarray):
    """Full-row softmax of S. Returns (P, m, l) with P = exp(S - m) / l."""
    m = S.max(axis=1)
    E = np.exp(S - m[:, None])
    l = E.sum(axis=1)
    return E / l[:, None], m, l


def _dscores(P: np.ndarray, dP: np.ndarray, delta: np.ndarray) -> np.ndarray:
    """dS = P * (dP - Delta 1^T): the softmax Jacobian applied to dP."""
    return P * (dP - delta[:, None])


def head_forward_backward(Q, K, V, dO, scale: float, block_rows: int = 512, check_rows: bool = False):
    """Attention forward and backward for one (sequence, head): Q, dO [Lq, D]; K, V [Lk, D]
    (Lk = Lq = L for self-attention).

    Returns float64 (O [Lq,D], lse [Lq], delta [Lq], dQ [Lq,D], dK [Lk,D], dV [Lk,D]).
    """
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    dO = np.asarray(dO, dtype=np.float64)
    L, D = Q.shape
    Lk = K.shape[0]
    if L > 0 and Lk == 0:
        raise ValueError("a sequence with queries but no keys has no softmax")
    O = np.zeros((L, D))
    lse = np.zeros(L)
    delta = np.zeros(L)
    dQ = np.zeros((L, D))
    dK = np.zeros((Lk, D))
    dV = np.zeros((Lk, D))
    if L == 0:
        return O, lse, delta, dQ, dK, dV
    block_rows = max(1, int(block_rows))
    for r0 in range(0, L, block_rows):
        r1 = min(L, r0 + block_rows)
        Qb, dOb = Q[r0:r1], dO[r0:r1]
        S = _scores(Qb, K, scale)
        P, m, l = _row_softmax(S)
        if check_rows:
            assert np.all(np.abs(P.sum(axis=1) - 1.0) <= 1e-12), "softmax rows do not sum to 1"
        Ob = P @ V
        O[r0:r1] = Ob
        lse[r0:r1] = m + np.log(l)
        db = np.sum(dOb * Ob, axis=1)
        delta[r0:r1] = db
        dV += P.T @ dOb
        dP = dOb @ V.T
        dS = _dscores(P, dP, db)
        dQ[r0:r1] = scale * (dS @ K)
        dK += scale * (dS.T @ Qb)
    return O, lse, delta, dQ, dK, dV


def _as_f64_thd(x):
    x = np.asarray(x)
    if x.ndim != 3:
        raise ValueError("tensors must be [T, H, D]")
    return x


def _check_cu(cu: np.ndarray, T: int, what: str):
    if cu.shape[0] < 1 or cu[0] != 0 or np.any(np.diff(cu) < 0) or cu[-1] != T:
        raise ValueError(f"bad {what}")


def attention(q, k, v, dout, cu_seqlens, scale: float, block_rows: int = 512,
              heads=None, check_rows: bool = False, cu_seqlens_k=None) -> dict:
    """Packed attention forward + backward over every sequence and the given heads.

    q, dout: float arrays [Tq, H, D]; k, v: [Tk, H, D], holding the exact bf16 input values.
    cu_seqlens: int [nseq + 1] query offsets, cu[0] = 0, non-decreasing; cu_seqlens_k: the
    key offsets (same nseq), or None for self-attention (cu_seqlens_k = cu_seqlens).
    Returns float64 arrays: out, dq [Tq, H, D]; dk, dv [Tk, H, D]; lse, delta [H, Tq].
    Heads not listed in ``heads`` are left at zero.
    """
    q, k, v, dout = (_as_f64_thd(a) for a in (q, k, v, dout))
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    cuk = cu if cu_seqlens_k is None else np.asarray(cu_seqlens_k, dtype=np.int64)
    T, H, D = q.shape
    Tk = k.shape[0]
    _check_cu(cu, T, "cu_seqlens")
    _check_cu(cuk, Tk, "cu_seqlens_k")
    if cuk.shape[0] != cu.shape[0]:
        raise ValueError("cu_seqlens and cu_seqlens_k differ in length")
    hs = range(H) if heads is None else list(heads)
    res = {
        "out": np.zeros((T, H, D)), "dq": np.zeros((T, H, D)),
        "dk": np.zeros((Tk, H, D)), "dv": np.zeros((Tk, H, D)),
        "lse": np.zeros((H, T)), "delta": np.zeros((H, T)),
    }
    for s in range(cu.shape[0] - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        ka, kb = int(cuk[s]), int(cuk[s + 1])
        if b == a:
            continue
        for h in hs:
            O, lse, dl, dQ, dK, dV = head_forward_backward(
                q[a:b, h], k[ka:kb, h], v[ka:kb, h], dout[a:b, h], scale, block_rows, check_rows)
            res["out"][a:b, h] = O
            res["dq"][a:b, h] = dQ
            res["dk"][ka:kb, h] = dK
            res["dv"][ka:kb, h] = dV
            res["lse"][h, a:b] = lse
            res["delta"][h, a:b] = dl
    return res


def _seq_of(cu: np.ndarray, t: int) -> int:
    return int(np.searchsorted(cu, t, side="right") - 1)


def query_rows(q, k, v, dout, cu_seqlens, scale: float, tokens, heads, cu_seqlens_k=None) -> dict:
    """Exact out, lse and dq for individual (query token, head) pairs.

    Each pair needs only its own score row over its sequence's keys: O(Lk * D)
    work, so this scales to the full-size workloads. Returns float64 arrays with
    one row per pair: out [n, D], lse [n], dq [n, D].
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    cuk = cu if cu_seqlens_k is None else np.asarray(cu_seqlens_k, dtype=np.int64)
    n = len(tokens)
    D = q.shape[2]
    out = np.zeros((n, D))
    lse = np.zeros(n)
    dq = np.zeros((n, D))
    for i, (t, h) in enumerate(zip(tokens, heads)):
        t, h = int(t), int(h)
        s = _seq_of(cu, t)
        a, b = int(cuk[s]), int(cuk[s + 1])
        qi = np.asarray(q[t, h], dtype=np.float64)[None, :]
        K = np.asarray(k[a:b, h], dtype=np.float64)
        V = np.asarray(v[a:b, h], dtype=np.float64)
        dOi = np.asarray(dout[t, h], dtype=np.float64)[None, :]
        S = _scores(qi, K, scale)
        P, m, l = _row_softmax(S)
        Oi = P @ V
        di = np.sum(dOi * Oi, axis=1)
        dS = _dscores(P, dOi @ V.T, di)
        out[i] = Oi[0]
        lse[i] = m[0] + np.log(l[0])
        dq[i] = scale * (dS @ K)[0]
    return {"out": out, "lse": lse, "dq": dq}


def key_rows(q, k, v, dout, cu_seqlens, scale: float, seq: int, head: int, keys,
             block_rows: int = 1024, cu_seqlens_k=None) -> dict:
    """Exact dk and dv for chosen keys (indices within sequence ``seq``'s keys) of one head.

    Needs every query's full score row (for its normaliser and Delta), so it
    costs O(Lq * Lk * D) for the sequence; it keeps only the chosen key columns.
    Returns float64 dk [n, D], dv [n, D].
    """
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    cuk = cu if cu_seqlens_k is None else np.asarray(cu_seqlens_k, dtype=np.int64)
    a, b = int(cu[seq]), int(cu[seq + 1])
    ka, kb = int(cuk[seq]), int(cuk[seq + 1])
    keys = np.asarray(keys, dtype=np.int64)
    Q = np.asarray(q[a:b, head], dtype=np.float64)
    K = np.asarray(k[ka:kb, head], dtype=np.float64)
    V = np.asarray(v[ka:kb, head], dtype=np.float64)
    dO = np.asarray(dout[a:b, head], dtype=np.float64)
    L = b - a
    Vs = V[keys]
    dk = np.zeros((keys.shape[0], Q.shape[1]))
    dv = np.zeros((keys.shape[0], Q.shape[1]))
    for r0 in range(0, L, block_rows):
        r1 = min(L, r0 + block_rows)
        Qb, dOb = Q[r0:r1], dO[r0:r1]
        P, m, l = _row_softmax(_scores(Qb, K, scale))
        Ob = P @ V
        db = np.sum(dOb * Ob, axis=1)
        Pc = P[:, keys]
        dPc = dOb @ Vs.T
        dSc = _dscores(Pc, dPc, db)
        dv += Pc.T @ dOb
        dk += scale * (dSc.T @ Qb)
    return {"dk": dk, "dv": dv}


def key_rows_torch(q, k, v, dout, cu_seqlens, scale: float, seq: int, head: int, keys,
                   block_rows: int = 2048, cu_seqlens_k=None, progress=None) -> dict:
    """``key_rows`` with torch float64 CPU tensor operations (multithreaded matmul and exp).

    Same steps as ``key_rows``; used for the 75,600- and 100,800-token clips, where one
    head's full score matrix is about 10^10 entries. ``progress(r1, L)``, if given, is
    called after each block of query rows (long runs report how far they are).
    """
    import torch
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    cuk = cu if cu_seqlens_k is None else np.asarray(cu_seqlens_k, dtype=np.int64)
    a, b = int(cu[seq]), int(cu[seq + 1])
    ka, kb = int(cuk[seq]), int(cuk[seq + 1])
    kt = torch.as_tensor(np.asarray(keys, dtype=np.int64))

    def t64(x, r0, r1):
        return torch.as_tensor(np.ascontiguousarray(np.asarray(x[r0:r1, head], dtype=np.float64)))

    Q, K, V, dO = t64(q, a, b), t64(k, ka, kb), t64(v, ka, kb), t64(dout, a, b)
    L = b - a
    Vs = V[kt]
    dk = torch.zeros((kt.shape[0], Q.shape[1]), dtype=torch.float64)
    dv = torch.zeros_like(dk)
    for r0 in range(0, L, block_rows):
        r1 = min(L, r0 + block_rows)
        Qb, dOb = Q[r0:r1], dO[r0:r1]
        S = scale * (Qb @ K.T)
        m = S.max(dim=1).values
        E = torch.exp(S - m[:, None])
        P = E / E.sum(dim=1)[:, None]
        Ob = P @ V
        db = (dOb * Ob).sum(dim=1)
        Pc = P[:, kt]
        dSc = Pc * (dOb @ Vs.T - db[:, None])
        dv += Pc.T @ dOb
        dk += scale * (dSc.T @ Qb)
        if progress is not None:
            progress(r1, L)
    return {"dk": dk.numpy(), "dv": dv.numpy()}
