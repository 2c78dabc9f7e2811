"""torch.autograd wrappers over the C ABI: attention and projection products
usable inside an ordinary training step.  Argument marshalling only -- every
forward and backward runs in the library's kernels (fbl_attn_fwd /
fbl_attn_bwd, fbl_proj); torch provides the tensors, the stream and the
autograd graph.

  attention(q, k, v, Hq, Hkv, scale=None, causal=False, kv_len=None) -> O
      q [B, S_q, Hq*d], k and v [B, S_kv, Hkv*d], token-major (any row
      stride, inner stride 1); gradients flow to q, k and v.
  attention_packed(qkv, Hq, Hkv, scale=None, causal=False) -> O
      qkv [B, S, (Hq + 2 Hkv) d], the packed output of a fused QKV
      projection; its gradient is one packed tensor of the same shape.
  linear(x, w) -> x @ w
      x [..., K] (rows contiguous), w [K, N]; gradients x and w by the data-
      and weight-gradient products, no transposed copy of either.

The incoming gradient is read in place, never copied: it must have unit
inner stride (any row stride), like every tensor the kernels read.  Autograd
can hand over a broadcast view (the gradient of a plain .sum(), inner stride
0); such a gradient is rejected with FblError, and the caller makes it
contiguous (or backpropagates a materialised tensor) instead.
"""
import math

import torch

from . import fbl as _f


def _unit(t, what: str):
    """The incoming gradient as it is, if its rows have unit inner stride."""
    if t.dim() == 0 or t.stride(-1) != 1:
        raise _f.FblError(_f.FBL_ERR_LAYOUT, f"{what}: the incoming gradient needs unit inner stride, got strides "
                                             f"{tuple(t.stride())}; pass a contiguous gradient")
    return t


class _Attention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, Hq, Hkv, scale, causal, kv_len):
        o, lse = _f.attn_fwd(q, k, v, Hq, Hkv, scale, causal, kv_len)
        ctx.save_for_backward(q, k, v, o, lse, kv_len if kv_len is not None else torch.empty(0))
        ctx.cfg = (Hq, Hkv, scale, causal, kv_len is not None)
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse, kv = ctx.saved_tensors
        Hq, Hkv, scale, causal, has_kv = ctx.cfg
        dq, dk, dv = _f.attn_bwd(q, k, v, o, _unit(do, 'attention'), lse, Hq, Hkv, scale, causal,
                                 kv if has_kv else None)
        return dq, dk, dv, None, None, None, None, None


def attention(q, k, v, Hq: int, Hkv: int, scale=None, causal: bool = False, kv_len=None):
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1] // Hq)
    return _Attention.apply(q, k, v, Hq, Hkv, float(scale), bool(causal), kv_len)


class _AttentionPacked(torch.autograd.Function):
    @staticmethod
    def forward(ctx, qkv, Hq, Hkv, scale, causal):
        o, lse = _f.attn_fwd_packed(qkv, Hq, Hkv, scale, causal)
        ctx.save_for_backward(qkv, o, lse)
        ctx.cfg = (Hq, Hkv, scale, causal)
        return o

    @staticmethod
    def backward(ctx, do):
        qkv, o, lse = ctx.saved_tensors
        Hq, Hkv, scale, causal = ctx.cfg
        dqkv = _f.attn_bwd_packed(qkv, o, _unit(do, 'attention_packed'), lse, Hq, Hkv, scale, causal)
        return dqkv, None, None, None, None


def attention_packed(qkv, Hq: int, Hkv: int, scale=None, causal: bool = False):
    if scale is None:
        scale = 1.0 / math.sqrt(qkv.shape[-1] // (Hq + 2 * Hkv))
    return _AttentionPacked.apply(qkv, Hq, Hkv, float(scale), bool(causal))


class _Linear(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w):
        x2 = x.reshape(-1, x.shape[-1])  # a view for token-major activations
        y = _f.proj(_f.FBL_PROJ_FWD, x2, w)
        ctx.save_for_backward(x2, w)
        ctx.xshape = x.shape
        return y.view(*x.shape[:-1], w.shape[1])

    @staticmethod
    def backward(ctx, dy):
        x2, w = ctx.saved_tensors
        dy = _unit(dy, "linear")
        try:
            dy2 = dy.view(-1, dy.shape[-1])  # a view: token rows of the incoming gradient
        except RuntimeError as e:
            raise _f.FblError(_f.FBL_ERR_LAYOUT, f"linear: the incoming gradient's rows are not one strided "
                                                 f"matrix ({e}); pass a contiguous gradient") from None
        dx = dw = None
        if ctx.needs_input_grad[0]:
            dx = _f.proj(_f.FBL_PROJ_BWD_DATA, dy2, w).view(ctx.xshape)
        if ctx.needs_input_grad[1]:
            dw = _f.proj(_f.FBL_PROJ_BWD_WEIGHT, x2, dy2)
        return dx, dw


def linear(x, w):
    return _Linear.apply(x, w)
