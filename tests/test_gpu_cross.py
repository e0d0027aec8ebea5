"""Cross-attention (queries and keys from separate token streams, t2v_attn_fwd_qk /
t2v_attn_bwd_qk) vs the float64 oracle: small packs element by element (several tiles on
both sides, ragged tails, empty sequences), the self-attention special case bitwise against
t2v_attn_fwd / t2v_attn_bwd, a closed form, and the cross workload at full size (sampled
query rows and key columns, per-(sequence, head) invariants)."""
import zlib

import numpy as np
import pytest

import oracle
from paper_2607_01701_amd.workload import bf16_bits_to_f32, make_pack, make_pack_qk, make_workload

from gpu_util import TOL_LSE, TOL_REL, assert_within, compare_full, dev_inputs, log, run_hip, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def oracle_of(pack):
    return oracle.attention(pack.f32("q"), pack.f32("k"), pack.f32("v"), pack.f32("dout"), pack.cu_seqlens,
                            pack.scale, cu_seqlens_k=pack.cu_seqlens_k)


CROSS = [
    ("cross_edges_d128", [1, 63, 65, 1000, 2000, 129], [1, 77, 256, 300, 129, 64], 2, 128),
    ("cross_edges_d64", [1, 63, 65, 1000, 2000, 129], [1, 77, 256, 300, 129, 64], 2, 64),
    ("cross_long_keys", [5, 33, 300], [3000, 700, 31], 2, 128),
    ("cross_empty_sequences", [0, 100, 0, 7], [0, 50, 0, 300], 3, 128),
]


@pytest.mark.parametrize("name,lq,lk,H,D", CROSS, ids=[c[0] for c in CROSS])
def test_parity_cross_packs(name, lq, lk, H, D):
    pack = make_pack_qk(lq, lk, H, D, seed=zlib.crc32(name.encode()) % 1000)
    log(f"case {name} lq={lq} lk={lk} H={H} D={D}")
    g = to_np(run_hip(pack))
    ref = oracle_of(pack)
    errs, _ = compare_full(g, ref, pack.cu_seqlens, name, cu_k=pack.cu_seqlens_k)
    assert_within(errs)


def test_self_case_matches_self_entry_points_bitwise():
    """t2v_attn_fwd_qk / _bwd_qk with equal offsets give exactly what t2v_attn_fwd / _bwd give."""
    import torch
    lens = [300, 65, 1000, 1]
    pack = make_pack(lens, 2, 128, seed=31)
    log("case self via qk entry points")
    d = dev_inputs(pack)
    a = run_hip(pack, d)
    pack.cu_seqlens_k = pack.cu_seqlens.copy()  # a distinct array with the same offsets
    b = run_hip(pack, d)
    for k in a:
        assert torch.equal(a[k], b[k]), k


def test_cross_deterministic_bitwise():
    import torch
    pack = make_pack_qk([700, 129], [200, 1000], 2, 128, seed=32)
    log("case cross determinism")
    d = dev_inputs(pack)
    a = run_hip(pack, d)
    b = run_hip(pack, d)
    for k in a:
        assert torch.equal(a[k], b[k]), k


def test_cross_one_key_closed_form():
    """One key per sequence: every query's output is that key's V row; dv = sum of dout."""
    pack = make_pack_qk([300, 70], [1, 1], 2, 128, seed=33)
    log("case cross one key")
    g = to_np(run_hip(pack))
    v = pack.f32("v").astype(np.float64)
    do = pack.f32("dout").astype(np.float64)
    cq = pack.cu_seqlens
    for s in range(2):
        a, b = int(cq[s]), int(cq[s + 1])
        assert np.array_equal(g["out"][a:b], np.broadcast_to(v[s], (b - a,) + v.shape[1:]))
        ref = do[a:b].sum(axis=0)
        assert np.max(np.abs(g["dv"][s] - ref)) <= 2e-2 * np.max(np.abs(ref))
    assert np.max(np.abs(g["dq"])) <= 1e-3 and np.max(np.abs(g["dk"])) <= 1e-3


def test_cross_workload_full_size():
    """The cross workload (16 video clips, 1,280-20,280 tokens, against 32-256 text tokens, 12 x 128)
    in the launch configuration the benchmark times: sampled query rows (out, lse, dq), all keys of
    one head of the longest clip (dk, dv), and per-(sequence, head) invariants."""
    import torch
    pack = make_workload("cross")
    log(f"case cross workload: Tq={pack.total_tokens} Tk={pack.total_tokens_k} H={pack.heads}")
    res = run_hip(pack)
    cq, ck = pack.cu_seqlens, pack.cu_seqlens_k
    q, k, v, do = (bf16_bits_to_f32(getattr(pack, n)).astype(np.float64) for n in ("q", "k", "v", "dout"))
    rng = np.random.default_rng(2)
    toks = np.concatenate([cq[:-1], cq[1:] - 1, rng.integers(0, pack.total_tokens, 24)])
    heads = rng.integers(0, pack.heads, toks.shape[0])
    ref = oracle.query_rows(q, k, v, do, cq, pack.scale, toks, heads, cu_seqlens_k=ck)
    ti, hi = torch.as_tensor(toks, device="cuda"), torch.as_tensor(heads, device="cuda")
    for name in ("out", "dq"):
        got = res[name][ti, hi].double().cpu().numpy()
        err = np.max(np.abs(got - ref[name])) / np.max(np.abs(ref[name]))
        log(f"  {name} sampled rel err {err:.2e}")
        assert err <= TOL_REL, name
    lse = res["lse"][hi, ti].double().cpu().numpy()
    assert np.max(np.abs(lse - ref["lse"])) <= TOL_LSE
    s = int(np.argmax(np.diff(cq)))
    h = 5
    nk = int(ck[s + 1] - ck[s])
    kr = oracle.key_rows(q, k, v, do, cq, pack.scale, seq=s, head=h, keys=np.arange(nk), cu_seqlens_k=ck)
    for name in ("dk", "dv"):
        got = res[name][int(ck[s]):int(ck[s + 1]), h].double().cpu().numpy()
        err = np.max(np.abs(got - kr[name])) / np.max(np.abs(kr[name]))
        log(f"  {name} clip {s} head {h} rel err {err:.2e}")
        assert err <= TOL_REL, name
    # invariants for every (sequence, head)
    dq, dk, dv = (res[n].double().cpu().numpy() for n in ("dq", "dk", "dv"))
    for si in range(len(cq) - 1):
        a, b, ka, kb = int(cq[si]), int(cq[si + 1]), int(ck[si]), int(ck[si + 1])
        sdk = np.abs(dk[ka:kb].sum(axis=0)).max(axis=1)
        mag = np.abs(dk[ka:kb]).sum(axis=0).max(axis=1)
        assert np.all(sdk <= 5e-3 * mag + 1e-6), si
        ddv = np.abs(dv[ka:kb].sum(axis=0) - do[a:b].sum(axis=0)).max(axis=1)
        assert np.all(ddv <= 1e-3 * np.abs(do[a:b]).sum(axis=0).max(axis=1) + 1e-6), si
        lq = np.einsum("thd,thd->h", q[a:b], dq[a:b])
        lk = np.einsum("thd,thd->h", k[ka:kb], dk[ka:kb])
        den = np.einsum("thd->h", np.abs(q[a:b] * dq[a:b])) + np.einsum("thd->h", np.abs(k[ka:kb] * dk[ka:kb]))
        assert np.all(np.abs(lq - lk) <= 5e-3 * den + 1e-6), si
