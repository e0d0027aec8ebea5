"""PyTorch autograd wrapper over the C ABI: the forward calls t2v_attn_fwd (or _qk), the
backward t2v_attn_bwd (or _qk) with the saved out and lse, so a training step (the DiT
forward and backward of Fig. 1) can use the library through loss.backward(). Argument
marshalling only; every step runs in the HIP library."""
from __future__ import annotations

import numpy as np

from ._lib import _cu_array, attn_bwd, attn_fwd


def _function():
    import torch

    class _VarlenAttention(torch.autograd.Function):
        @staticmethod
        def forward(ctx, q, k, v, cu_seqlens, scale, cu_seqlens_k):
            out, lse = attn_fwd(q, k, v, cu_seqlens, scale, cu_seqlens_k=cu_seqlens_k)
            ctx.save_for_backward(q, k, v, out, lse)
            ctx.cu, ctx.cu_k, ctx.scale = cu_seqlens, cu_seqlens_k, scale
            ctx.mark_non_differentiable(lse)
            return out, lse

        @staticmethod
        def backward(ctx, dout, _dlse):
            q, k, v, out, lse = ctx.saved_tensors
            dq, dk, dv = attn_bwd(q, k, v, out, lse, dout.contiguous(), ctx.cu, ctx.scale, cu_seqlens_k=ctx.cu_k)
            return dq, dk, dv, None, None, None

    return _VarlenAttention


_FN = None


def varlen_attention(q, k, v, cu_seqlens, scale: float, cu_seqlens_k=None):
    """Packed variable-length attention with autograd: q [Tq, H, D], k, v [Tk, H, D] bf16 on the
    GPU; cu_seqlens (and cu_seqlens_k for cross-attention) host int32 offsets. Returns (out, lse);
    gradients flow to q, k and v (lse is not differentiated)."""
    global _FN
    if _FN is None:
        _FN = _function()
    cu = _cu_array(cu_seqlens)
    ck = None if cu_seqlens_k is None else _cu_array(cu_seqlens_k)
    return _FN.apply(q, k, v, np.array(cu, copy=True), float(scale), None if ck is None else np.array(ck, copy=True))
