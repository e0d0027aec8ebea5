"""Seeded random packs on the GPU, element by element against the float64 oracle: self- and
cross-attention, 1-6 heads, head_dim 64 and 128, empty and one-token sequences, long query
segments against short key segments. Few heads and uneven lengths reach every scheduling
path: whole-group and single-item XCD dealing, narrow and wide tiles, and the dK/dV loop
split (checked to occur in at least one pack)."""
import numpy as np
import pytest

import oracle
from paper_2607_01701_amd.workload import make_pack, make_pack_qk

from gpu_util import assert_within, compare_full, log, run_hip, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def random_pack(seed):
    rng = np.random.default_rng(1000 + seed)
    nseq = int(rng.integers(1, 9))
    heads = int(rng.integers(1, 7))
    D = 64 if rng.random() < 0.4 else 128
    kind = ("self", "cross", "split")[seed % 3]
    if kind == "self":
        lens = [int(x) for x in rng.choice([0, 1, 31, 64, 65, 255, 257, 700, 1500, 3000], size=nseq)]
        if sum(lens) == 0:
            lens[0] = 129
        return make_pack(lens, heads, D, seed=seed), kind
    lq = [int(x) for x in rng.integers(1, 2500, size=nseq)]
    lk = [int(x) for x in rng.integers(1, 300, size=nseq)]
    if kind == "split":  # one long query segment against a short key segment
        lq[0], lk[0] = int(rng.integers(5000, 9000)), int(rng.integers(1, 129))
    for s in range(nseq):
        if rng.random() < 0.15:
            lq[s] = lk[s] = 0
    if sum(lq) == 0:
        lq[0], lk[0] = 100, 20
    return make_pack_qk(lq, lk, heads, D, seed=seed), kind


@pytest.mark.parametrize("seed", range(12))
def test_random_pack_matches_oracle(seed, monkeypatch, capfd):
    pack, kind = random_pack(seed)
    lq = np.diff(pack.cu_seqlens).tolist()
    lk = None if pack.cu_seqlens_k is None else np.diff(pack.cu_seqlens_k).tolist()
    log(f"case seed {seed} {kind}: H={pack.heads} D={pack.head_dim} lq={lq} lk={lk}")
    monkeypatch.setenv("T2V_LOG", "1")
    g = to_np(run_hip(pack))
    plans = capfd.readouterr().err
    ref = oracle.attention(pack.f32("q"), pack.f32("k"), pack.f32("v"), pack.f32("dout"), pack.cu_seqlens,
                           pack.scale, cu_seqlens_k=pack.cu_seqlens_k)
    errs, _ = compare_full(g, ref, pack.cu_seqlens, f"seed {seed}", cu_k=pack.cu_seqlens_k)
    assert_within(errs)
    if kind == "split":  # a 5,000-9,000-query loop against few key tiles: the dK/dV loop is split
        assert "loops split at" in plans, plans
