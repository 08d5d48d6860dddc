"""torch.autograd functions over the C ABI: the fused attention (and its
block-sparse and bias / relu forms) as differentiable operations for training
code.

``attention`` runs attnfuse_fwd, keeps Q, K, V, O and the row statistic LSE
(Section 4.4: the forward saves one scalar per row), and its backward runs
attnfuse_bwd on the incoming gradient of O.  Argument marshalling only: every
step of the computation runs in the HIP kernels, and the gradients are exactly
those attnfuse_bwd returns.  ALiBi slopes, theta, the window and the scale get
no gradient.
"""
import torch

from . import api


class _Attention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, alibi_slopes, rope, theta, mask, window, scale):
        o, lse = api.attnfuse_fwd(q, k, v, rope=rope, theta=theta, mask=mask, window=window,
                                  alibi_slopes=alibi_slopes, scale=scale)
        ctx.save_for_backward(q, k, v, o, lse, alibi_slopes)
        ctx.cfg = dict(rope=rope, theta=theta, mask=mask, window=window, scale=scale)
        ctx.mark_non_differentiable(lse)
        return o, lse

    @staticmethod
    def backward(ctx, do, _dlse):
        q, k, v, o, lse, slopes = ctx.saved_tensors
        dq, dk, dv = api.attnfuse_bwd(q, k, v, o, do.contiguous(), lse, alibi_slopes=slopes, **ctx.cfg)
        return dq, dk, dv, None, None, None, None, None, None


class _BlockSparseAttention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, alibi_slopes, block_mask, rope, theta, mask, window, scale):
        o, lse = api.attnfuse_fwd_blocksparse(q, k, v, block_mask, rope=rope, theta=theta, mask=mask, window=window,
                                              alibi_slopes=alibi_slopes, scale=scale)
        ctx.save_for_backward(q, k, v, o, lse, alibi_slopes)
        ctx.block_mask = block_mask
        ctx.cfg = dict(rope=rope, theta=theta, mask=mask, window=window, scale=scale)
        ctx.mark_non_differentiable(lse)
        return o, lse

    @staticmethod
    def backward(ctx, do, _dlse):
        q, k, v, o, lse, slopes = ctx.saved_tensors
        dq, dk, dv = api.attnfuse_bwd_blocksparse(q, k, v, o, do.contiguous(), lse, ctx.block_mask,
                                                  alibi_slopes=slopes, **ctx.cfg)
        return dq, dk, dv, None, None, None, None, None, None, None


class _BiasNormAttention(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, bias, norm, rope, theta, mask, window, scale):
        o, lse = api.attnfuse_fwd_bias_norm(q, k, v, bias=bias, norm=norm, rope=rope, theta=theta, mask=mask,
                                            window=window, scale=scale)
        ctx.save_for_backward(q, k, v, o, lse, bias)
        ctx.cfg = dict(norm=norm, rope=rope, theta=theta, mask=mask, window=window, scale=scale)
        if lse is not None:
            ctx.mark_non_differentiable(lse)
        return o, lse

    @staticmethod
    def backward(ctx, do, _dlse):
        q, k, v, o, lse, bias = ctx.saved_tensors
        dq, dk, dv = api.attnfuse_bwd_bias_norm(q, k, v, o, do.contiguous(), lse, bias=bias, **ctx.cfg)
        return dq, dk, dv, None, None, None, None, None, None, None


def attention(q, k, v, *, rope="none", theta=10000.0, mask="causal", window=None, alibi_slopes=None, scale=None,
              return_lse=False):
    """Differentiable fused attention: O [B, H, S, D] (and the non-differentiable
    LSE [B, H, S] with ``return_lse``); arguments as api.attnfuse_fwd."""
    o, lse = _Attention.apply(q, k, v, alibi_slopes, rope, theta, mask, window, scale)
    return (o, lse) if return_lse else o


def blocksparse_attention(q, k, v, block_mask, *, rope="none", theta=10000.0, mask="none", window=None,
                          alibi_slopes=None, scale=None, return_lse=False):
    """Differentiable block-sparse attention over a blockmask.BlockMask;
    arguments as api.attnfuse_fwd_blocksparse."""
    o, lse = _BlockSparseAttention.apply(q, k, v, alibi_slopes, block_mask, rope, theta, mask, window, scale)
    return (o, lse) if return_lse else o


def attention_bias_norm(q, k, v, *, bias=None, norm="softmax", rope="none", theta=10000.0, mask="causal",
                        window=None, scale=None, return_lse=False):
    """Differentiable attention with a dense additive bias tensor and softmax or
    relu normalisation; arguments as api.attnfuse_fwd_bias_norm (the bias gets
    no gradient; under relu attention LSE is None)."""
    o, lse = _BiasNormAttention.apply(q, k, v, bias, norm, rope, theta, mask, window, scale)
    return (o, lse) if return_lse else o
