"""The largest head count the boundary accepts: H * D = 2^22 (the validation limit, rows of
8 MiB), at D = 128 (32,768 heads) and D = 64 (65,536 heads), on a ragged pack of three
clips. Inputs are drawn on the GPU from a seeded generator (about 1.4 GB per tensor at this
size, too slow to draw on the host). The float64 oracle checks a spread of heads, including
the last, whose elements sit at the highest offsets of every row; a head permutation of the
inputs must permute every output bitwise, which checks the indexing of all heads."""
import numpy as np
import pytest

import oracle

from gpu_util import assert_within, compare_full, log

pytestmark = pytest.mark.gpu

LENS = [1, 33, 130]  # one-token clip, one partial tile, two tiles with a ragged tail


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _draw(shape, gen):
    import torch
    return torch.randn(shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)


def _run(d, cu, scale):
    import torch
    from paper_2607_01701_amd import attn_bwd, attn_fwd
    out, lse = attn_fwd(d["q"], d["k"], d["v"], cu, scale)
    dq, dk, dv = attn_bwd(d["q"], d["k"], d["v"], out, lse, d["dout"], cu, scale)
    torch.cuda.synchronize()
    return {"out": out, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


@pytest.mark.parametrize("D", [128, 64])
def test_largest_head_count(D):
    import torch
    H = (1 << 22) // D
    cu = np.concatenate([[0], np.cumsum(LENS)]).astype(np.int32)
    T = int(cu[-1])
    scale = 1.0 / float(np.sqrt(D))
    log(f"case largest head count H={H} D={D} lens={LENS} ({T * H * D * 2 / 2**30:.2f} GiB per tensor)")
    gen = torch.Generator(device="cuda")
    gen.manual_seed(4242 + D)
    d = {n: _draw((T, H, D), gen) for n in ("q", "k", "v", "dout")}
    g = _run(d, cu, scale)

    heads = [0, 1, H // 2, H - 2, H - 1]
    sub = {n: d[n][:, heads].float().cpu().numpy() for n in d}
    ref = oracle.attention(sub["q"], sub["k"], sub["v"], sub["dout"], cu, scale)
    got = {n: g[n][:, heads].float().cpu().numpy().astype(np.float64) for n in ("out", "dq", "dk", "dv")}
    got["lse"] = g["lse"][heads].cpu().numpy().astype(np.float64)
    errs, _ = compare_full(got, ref, cu, f"H={H} D={D} heads {heads}")
    assert_within(errs)

    # Heads are independent: permuting the heads of every input permutes every output.
    perm = torch.randperm(H, generator=torch.Generator().manual_seed(7)).cuda()
    dp = {n: d[n].index_select(1, perm) for n in d}
    del d
    gp = _run(dp, cu, scale)
    for n in ("out", "dq", "dk", "dv"):
        assert torch.equal(gp[n], g[n].index_select(1, perm)), n
    assert torch.equal(gp["lse"], g["lse"].index_select(0, perm)), "lse"
    log(f"H={H} D={D}: head permutation equivariant bitwise over all heads")
