"""Numerical edge cases of the HIP path against the float64 oracle: scores that rise on
every 32-key step (the online softmax's reference maximum moves on each step), extreme
finite logits (near one-hot softmax), the 30-head x 64 shape of Table II at a mid size, and
NaN propagation (a NaN query row poisons exactly what the definition says it must)."""
import numpy as np
import pytest

import oracle
from paper_2607_01701_amd.workload import bf16_bits_to_f32, f32_to_bf16_bits, make_pack

from gpu_util import assert_within, compare_full, dev_inputs, log, run_hip, to_np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def oracle_of(pack):
    return oracle.attention(pack.f32("q"), pack.f32("k"), pack.f32("v"), pack.f32("dout"), pack.cu_seqlens,
                            pack.scale)


def rising_pack(lengths, H, D, seed, growth):
    """Keys whose score against every query rises linearly with the key position: the
    scaled score of key j is about growth * j / 32 natural units above key 0 (offsets
    centred on the clip), so with growth * log2(e) > 8 each 32-key step's maximum exceeds
    the previous one by more than the lazy-rescale threshold."""
    pack = make_pack(lengths, H, D, seed=seed)
    q = 0.25 * pack.f32("q") + 1.0
    k = pack.f32("k") * 0.25
    cu = pack.cu_seqlens
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        j = np.arange(b - a, dtype=np.float32)[:, None, None] - (b - a - 1) / 2.0
        # q . (1, ..., 1) ~ D: adding x * (1, ..., 1) to key j raises its scaled score by ~ x * D * scale.
        k[a:b] += (growth / 32.0) * j / (D * pack.scale)
    pack.q, pack.k = f32_to_bf16_bits(q), f32_to_bf16_bits(k)
    return pack


def dq_error_of_bf16_ds(pack, ref):
    """Relative max error of dq when only dS is rounded to bf16 (everything else exact):
    the precision floor of any backward that feeds dS to a bf16 product, as the kernels do."""
    q, k, v, do = (pack.f32(n).astype(np.float64) for n in ("q", "k", "v", "dout"))
    sc, cu = pack.scale, pack.cu_seqlens
    dq = np.zeros_like(ref["dq"])
    for s in range(len(cu) - 1):
        a, b = int(cu[s]), int(cu[s + 1])
        for h in range(pack.heads):
            p = np.exp(sc * q[a:b, h] @ k[a:b, h].T - ref["lse"][h, a:b][:, None])
            ds = p * (do[a:b, h] @ v[a:b, h].T - np.sum(do[a:b, h] * (p @ v[a:b, h]), axis=1)[:, None])
            dq[a:b, h] = sc * bf16_bits_to_f32(f32_to_bf16_bits(ds.astype(np.float32))).astype(np.float64) @ k[a:b, h]
    return float(np.max(np.abs(dq - ref["dq"])) / np.max(np.abs(ref["dq"])))


@pytest.mark.parametrize("D", [128, 64])
def test_reference_moves_every_step(D):
    pack = rising_pack([256, 160, 33], 2, D, seed=41, growth=7.0)
    log(f"case rising scores D={D}")
    g = to_np(run_hip(pack))
    ref = oracle_of(pack)
    # Query 0 of the 256-token clip: each 32-key step's maximum score is more than the
    # lazy-rescale threshold (8 in log2 units) above the previous step's.
    sq, sk = pack.f32("q")[:256, 0].astype(np.float64), pack.f32("k")[:256, 0].astype(np.float64)
    smax = (pack.scale * np.log2(np.e)) * (sq[0] @ sk.T)
    step_max = np.array([smax[i:i + 32].max() for i in range(0, 256, 32)])
    assert np.all(np.diff(step_max) > 8.0)
    errs, worst = compare_full(g, ref, pack.cu_seqlens, f"rising D={D}")
    # Near one-hot rows make dq a cancelling sum of dS times keys with a large shared part,
    # so bf16 rounding of dS alone costs ~1% here (logged); every output, dq included, is
    # still held to the usual bounds (measured dq 1.83e-2 at D = 128, 1.79e-2 at 64; the
    # kernels are deterministic, so these inputs always give the same errors).
    floor = dq_error_of_bf16_ds(pack, ref)
    log(f"  dq error with only dS rounded to bf16: {floor:.3e}")
    assert errs["dq"] >= 0.5 * floor, (errs["dq"], floor)  # the inputs do stress dq as intended
    assert_within(errs)


def test_extreme_logits():
    """Scores in the hundreds of natural units: softmax rows are near one-hot."""
    pack = make_pack([700, 129, 2], 2, 128, seed=43)
    pack.q = f32_to_bf16_bits(pack.f32("q") * 12.0)
    pack.k = f32_to_bf16_bits(pack.f32("k") * 12.0)
    log("case extreme logits")
    g = to_np(run_hip(pack))
    ref = oracle_of(pack)
    spread = ref["lse"].max() - ref["lse"].min()
    log(f"  lse range {ref['lse'].min():.1f} .. {ref['lse'].max():.1f}")
    assert spread > 100.0
    errs, worst = compare_full(g, ref, pack.cu_seqlens, "extreme logits")
    assert_within(errs)


def test_table2_head_shape_d64():
    """30 heads x 64 (the 1,920-wide model of Table II) over several tiles of a 4,096-token
    clip, a 1,280-token clip and a ragged 333-token one."""
    pack = make_pack([4096, 1280, 333], 30, 64, seed=44)
    log("case 30 x 64 mid-size")
    g = to_np(run_hip(pack))
    ref = oracle_of(pack)
    errs, worst = compare_full(g, ref, pack.cu_seqlens, "30x64")
    assert_within(errs)
    for k, e in worst.items():
        assert e <= 2e-2, (k, e)


def test_nan_query_row_propagation():
    """A NaN in one query row of clip 1, head 0: that row's out, lse and dq are NaN, so are
    dk and dv of every key of clip 1 in head 0 (each key receives a term from the NaN row).
    Every other value is bitwise what the run without the NaN gives, except the other rows
    of the NaN row's 32-query block in head 0: they share a wave, whose rescale decisions
    are taken together, so they may settle on another (equally valid) reference maximum
    and differ by rounding only."""
    import torch
    pack = make_pack([300, 257, 90], 2, 128, seed=45)
    clean = {k: v.clone() for k, v in run_hip(pack).items()}
    a, b = int(pack.cu_seqlens[1]), int(pack.cu_seqlens[2])
    row = a + 100
    bad = pack.q.copy()
    bad[row, 0, 5] = 0x7FC0  # bf16 quiet NaN
    pack.q = bad
    log(f"case NaN in q[{row}, head 0]")
    res = run_hip(pack)
    torch.cuda.synchronize()
    g = {k: v.float().cpu().numpy() for k, v in res.items()}
    c = {k: v.float().cpu().numpy() for k, v in clean.items()}
    expect = {k: np.zeros(g[k].shape, dtype=bool) for k in g}
    expect["out"][row, 0] = True
    expect["dq"][row, 0] = True
    expect["lse"][0, row] = True
    expect["dk"][a:b, 0] = True
    expect["dv"][a:b, 0] = True
    blk0 = a + ((row - a) // 32) * 32  # the NaN row's 32-query block (one wave)
    near = {k: np.zeros(g[k].shape, dtype=bool) for k in g}
    for k in ("out", "dq"):
        near[k][blk0:blk0 + 32, 0] = True
    near["lse"][0, blk0:blk0 + 32] = True
    for k in ("out", "lse", "dq", "dk", "dv"):
        nan = np.isnan(g[k])
        assert np.array_equal(nan, expect[k]), f"{k}: NaN pattern differs ({int(nan.sum())} vs {int(expect[k].sum())})"
        same = ~expect[k] & ~near[k]
        assert np.array_equal(g[k][same], c[k][same]), f"{k}: values outside the NaN row's block changed"
        blk = near[k] & ~expect[k]
        if blk.any():
            diff = float(np.max(np.abs(g[k][blk] - c[k][blk])))
            assert diff <= 2e-2 * float(np.max(np.abs(c[k][blk]))) + 1e-3, (k, diff)
