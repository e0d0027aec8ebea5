"""The C ABI on the GPU: offsets in device memory are refused before anything reads them.

cu_seqlens (and cu_seqlens_k) are read on the host by the scheduler; a device pointer must
return T2V_ERR_INVALID_ARG, not be dereferenced, and leave every output untouched. Each of
the four attention entry points is called with a torch device tensor's address as its
offsets (and, for the cross-attention calls, as each one of the two in turn)."""
import ctypes

import numpy as np
import pytest

from paper_2607_01701_amd import _lib
from paper_2607_01701_amd.workload import make_pack

from gpu_util import dev_inputs, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _ptr(addr):
    return ctypes.cast(ctypes.c_void_p(addr), _lib._i32p)


@pytest.mark.parametrize("entry", ["fwd", "bwd", "fwd_qk_q", "fwd_qk_k", "bwd_qk_q", "bwd_qk_k"])
def test_device_offsets_are_refused(entry):
    import torch
    log(f"case device cu_seqlens -> {entry}")
    pack = make_pack([100, 37], 2, 128, seed=3)
    d = dev_inputs(pack)
    T, H, D = pack.total_tokens, pack.heads, pack.head_dim
    cu_host = np.ascontiguousarray(pack.cu_seqlens, dtype=np.int32)
    cu_dev = torch.from_numpy(cu_host.copy()).cuda()
    outs = {n: torch.full((T, H, D), 3.0, dtype=torch.bfloat16, device="cuda") for n in ("out", "dq", "dk", "dv")}
    lse = torch.full((H, T), 5.0, dtype=torch.float32, device="cuda")
    ws = torch.full((2, H, T), 7.0, dtype=torch.float32, device="cuda")
    before = {n: t.clone() for n, t in outs.items()}
    lse0, ws0 = lse.clone(), ws.clone()
    torch.cuda.synchronize()
    L = _lib.lib()
    dp, hp = _ptr(cu_dev.data_ptr()), cu_host.ctypes.data_as(_lib._i32p)
    s = torch.cuda.current_stream().cuda_stream
    a = {n: d[n].data_ptr() for n in ("q", "k", "v", "dout")}
    sc = pack.scale
    if entry == "fwd":
        st = L.t2v_attn_fwd(a["q"], a["k"], a["v"], dp, 2, H, D, sc, outs["out"].data_ptr(), lse.data_ptr(), s)
    elif entry.startswith("fwd_qk"):
        cq, ck = (dp, hp) if entry.endswith("_q") else (hp, dp)
        st = L.t2v_attn_fwd_qk(a["q"], a["k"], a["v"], cq, ck, 2, H, D, sc, outs["out"].data_ptr(), lse.data_ptr(), s)
    elif entry == "bwd":
        st = L.t2v_attn_bwd(a["q"], a["k"], a["v"], a["q"], lse.data_ptr(), dp, 2, H, D, sc, a["dout"],
                            outs["dq"].data_ptr(), outs["dk"].data_ptr(), outs["dv"].data_ptr(), ws.data_ptr(), s)
    else:
        cq, ck = (dp, hp) if entry.endswith("_q") else (hp, dp)
        st = L.t2v_attn_bwd_qk(a["q"], a["k"], a["v"], a["q"], lse.data_ptr(), cq, ck, 2, H, D, sc, a["dout"],
                               outs["dq"].data_ptr(), outs["dk"].data_ptr(), outs["dv"].data_ptr(), ws.data_ptr(), s)
    msg = _lib.t2v_last_error(L)
    torch.cuda.synchronize()
    assert st == _lib.T2V_ERR_INVALID_ARG, (st, msg)
    assert "host pointer" in msg, msg
    for n in outs:
        assert torch.equal(outs[n], before[n]), f"{n} was written"
    assert torch.equal(lse, lse0) and torch.equal(ws, ws0), "lse or delta_ws was written"


def test_empty_pack_with_device_offsets_is_refused():
    """T = 0 returns early without launching, but only after the pointer check: a device
    array of one zero is still refused."""
    import torch
    L = _lib.lib()
    cu_dev = torch.zeros(1, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    st = L.t2v_attn_fwd(None, None, None, _ptr(cu_dev.data_ptr()), 0, 2, 128, 0.1, None, None, None)
    assert st == _lib.T2V_ERR_INVALID_ARG, _lib.t2v_last_error(L)
