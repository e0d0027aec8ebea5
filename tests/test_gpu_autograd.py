"""The autograd wrapper (varlen_attention) on the GPU: loss.backward() through it gives, bitwise,
the gradients of a direct t2v_attn_bwd call with the same dout, for self- and cross-attention;
and a two-layer toy step (attention feeding attention) backpropagates through both calls."""
import pytest

from paper_2607_01701_amd.workload import make_pack, make_pack_qk

from gpu_util import dev_inputs, log, run_hip

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


CASES = [
    ("self_d128", lambda: make_pack([1, 65, 300, 1000], 2, 128, seed=81)),
    ("self_d64", lambda: make_pack([257, 31], 3, 64, seed=82)),
    ("cross_d128", lambda: make_pack_qk([1000, 5, 129], [256, 3, 600], 2, 128, seed=83)),
]


@pytest.mark.parametrize("name,make", CASES, ids=[c[0] for c in CASES])
def test_backward_through_autograd_matches_the_direct_call(name, make):
    import torch
    from paper_2607_01701_amd import varlen_attention
    pack = make()
    d = dev_inputs(pack)
    log(f"case autograd {name}")
    want = run_hip(pack, d)
    q, k, v = (d[n].clone().requires_grad_(True) for n in ("q", "k", "v"))
    out, lse = varlen_attention(q, k, v, pack.cu_seqlens, pack.scale, cu_seqlens_k=pack.cu_seqlens_k)
    assert not lse.requires_grad
    (out.float() * d["dout"].float()).sum().backward()
    torch.cuda.synchronize()
    assert torch.equal(out.detach(), want["out"]) and torch.equal(lse, want["lse"])
    for t, n in ((q, "dq"), (k, "dk"), (v, "dv")):
        assert torch.equal(t.grad, want[n]), n


def test_two_layers_backpropagate():
    import torch
    from paper_2607_01701_amd import varlen_attention
    pack = make_pack([300, 77], 2, 128, seed=84)
    d = dev_inputs(pack)
    log("case autograd two layers")
    x = d["q"].clone().requires_grad_(True)
    h, _ = varlen_attention(x, d["k"], d["v"], pack.cu_seqlens, pack.scale)
    y, _ = varlen_attention(h, h, h, pack.cu_seqlens, pack.scale)
    y.float().square().mean().backward()
    torch.cuda.synchronize()
    assert x.grad is not None and torch.isfinite(x.grad.float()).all()
    assert float(x.grad.float().abs().max()) > 0.0
