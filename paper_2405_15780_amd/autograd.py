"""torch.autograd wrapper: attention as a differentiable op whose forward and
backward are the library's kernels (argument marshalling only).

attention(q, k, v) takes bf16 [B, H, Nq, d] queries and [B, H, Nk, d] keys
and values (any strides with d contiguous) and returns O in fp32. In the
backward, the upstream gradient is rounded to bf16 (the kernels' dO operand)
and dQ, dK, dV, computed in fp32, are returned in the inputs' dtype.
"""
from __future__ import annotations

from . import binding as _b


def _torch():
    import torch

    return torch


class _Attention:
    _fn = None

    @classmethod
    def get(cls):
        if cls._fn is None:
            torch = _torch()

            class Attention(torch.autograd.Function):
                @staticmethod
                def forward(ctx, q, k, v, scale, store_ds):
                    o, lse = _b.fwd(q, k, v, scale)
                    ctx.save_for_backward(q, k, v, o, lse)
                    ctx.scale, ctx.store_ds = scale, store_ds
                    return o

                @staticmethod
                def backward(ctx, grad_o):
                    q, k, v, o, lse = ctx.saved_tensors
                    dout = grad_o.to(torch.bfloat16)
                    if dout.stride(-1) != 1:
                        dout = dout.contiguous()
                    dq, dk, dv = _b.bwd(q, k, v, o, lse, dout, ctx.scale, store_ds=ctx.store_ds)
                    return dq.to(q.dtype), dk.to(k.dtype), dv.to(v.dtype), None, None

            cls._fn = Attention
        return cls._fn


def attention(q, k, v, scale=None, store_ds=False):
    """softmax(scale Q K^T) V (scale defaults to 1/sqrt(d)) with a backward
    pass; store_ds selects the dS mode of the backward."""
    return _Attention.get().apply(q, k, v, scale, store_ds)
