"""Input range of the bf16 path (through the C ABI).

* The backward's fp16 operands carry dO times a power of two chosen per
  (batch, K/V head), so gradients of any scale keep full precision: dO scaled
  by 2^-20 (typical of bf16 training without loss scaling) or by 2^20 gives
  gradients scaled by exactly the same factor, bit for bit, and both match the
  oracle.
* Queries and keys of norm ~1e3 (elements ~90, far above the usual range of
  activations, below fp16's maximum after rotation): the scores reach ~3e4
  and the softmax picks one key per row, so O is that key's value row and the
  gradients of Q and K vanish; LSE is checked against the bound that fp16
  rounding of the rotated operands puts on a score of that size.  (Scores of
  1e6, from elements of 1e3, are beyond fp32 itself: its resolution there is
  0.06, so re-deriving P = exp(s - LSE) in fp32 is only good to ~6%.)  The
  backward is handed the oracle's O and LSE (see test_gpu_bwd).
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, assert_bf16_close, bwd_refs, device_inputs, f64, given_lse, given_o, need_gpu
from paper_2609_13612_amd import api, inputs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rope,mask,D", [("neox", "causal", 128), ("none", "sliding_window", 64),
                                         ("interleaved", "none", 128)], ids=str)
@pytest.mark.parametrize("e", [-20, 20], ids=lambda e: f"2^{e}")
def test_bwd_dout_scale_exact(rope, mask, D, e):
    need_gpu()
    B, H, Hkv, S = 2, 8, 2, 300
    window = 90 if mask == "sliding_window" else None
    announce(f"dO scaled by 2^{e}: rope={rope} mask={mask} D={D}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=101, with_do=True)
    kw = dict(rope=rope, mask=mask, window=window)
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], **kw)
    g = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, **kw)
    do_s = (dev["do"].float() * 2.0 ** e).to(torch.bfloat16)   # exact: a power of two
    g_s = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, do_s, lse, **kw)
    torch.cuda.synchronize()
    for name, a, b in zip(("dQ", "dK", "dV"), g, g_s):
        assert torch.equal((b.float() * 2.0 ** -e).to(torch.bfloat16), a), f"{name}: not scaled exactly"
    ref = oracle.attention_backward(*[f64(cpu[n]) for n in ("q", "k", "v", "do")], **kw)
    for name, b, r in zip(("dQ", "dK", "dV"), g_s, ref):
        assert_bf16_close(f64(b) * 2.0 ** -e, r, f"{name} (dO x 2^{e}, rescaled)")


def test_bwd_small_dout_nonzero_everywhere():
    """Gradients of 1e-6 size: every visible key's dK and dV row is non-zero
    (fp16 operands without the scale would flush most of dS to zero)."""
    need_gpu()
    B, H, Hkv, S, D = 1, 4, 1, 512, 128
    announce("small dO: gradients not flushed")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=102, with_do=True)
    kw = dict(rope="neox", mask="causal")
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], **kw)
    do = (dev["do"].float() * 1e-6).to(torch.bfloat16)
    dq, dk, dv = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, do, lse, **kw)
    torch.cuda.synchronize()
    ref = oracle.attention_backward(*[f64(cpu[n]) for n in ("q", "k", "v")], f64(do.cpu()), **kw)
    for name, g, r in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref):
        gg = f64(g)
        # relative to the gradient's own size: 2e-2 of its largest element
        # (flushed products would leave errors of the order of the values)
        scale = float(np.abs(r).max())
        err = np.abs(gg - r)
        assert err.max() <= 2e-2 * scale and err.mean() <= 2e-3 * scale, \
            f"{name}: max {err.max():.3e} mean {err.mean():.3e} of max|ref| {scale:.3e}"


@pytest.mark.parametrize("rope", ["none", "neox"])
def test_large_query_key_magnitude(rope):
    need_gpu()
    B, H, Hkv, S, D = 1, 2, 1, 16, 128
    announce(f"|q|, |k| ~ 1e3 (norms), rope={rope}")
    g = torch.Generator("cpu").manual_seed(100)
    amp = 1000.0 / np.sqrt(D)                     # |q|, |k| ~ 1e3
    q = (amp * torch.randn(B, H, S, D, generator=g)).to(torch.bfloat16)
    k = (amp * torch.randn(B, Hkv, S, D, generator=g)).to(torch.bfloat16)
    v = torch.randn(B, Hkv, S, D, generator=g).to(torch.bfloat16)
    do = torch.randn(B, H, S, D, generator=g).to(torch.bfloat16)
    kw = dict(rope=rope, theta=10000.0, mask="none")
    fq, fk, fv, fdo = f64(q), f64(k), f64(v), f64(do)
    O, L = oracle.attention_forward(fq, fk, fv, **kw)
    o_ref, o_dev = given_o(O)
    o, lse = api.attnfuse_fwd(q.cuda(), k.cuda(), v.cuda(), **kw)
    # the backward is handed the oracle's forward output (see test_gpu_bwd)
    dq, dk, dv = api.attnfuse_bwd(q.cuda(), k.cuda(), v.cuda(), o_dev, do.cuda(), given_lse(L), **kw)
    torch.cuda.synchronize()
    scale = D ** -0.5
    pos = np.arange(S, dtype=np.float64)
    qr = oracle.rope_rotate(fq, pos, 10000.0, rope)
    kr = oracle.rope_rotate(fk, pos, 10000.0, rope)
    s = scale * np.einsum("bhmd,bnd->bhmn", qr, kr[:, 0])
    # a score's error: fp16 rounding of each rotated operand (2^-11 relative
    # each; none without RoPE, whose bf16 operands are exact) and fp32
    # accumulation over D terms (below 2^-16 relative to sum_d |q'_d k'_d|)
    rel = (2 * 2.0 ** -11 if rope != "none" else 0.0) + 2.0 ** -16
    bound = scale * np.einsum("bhmd,bnd->bhmn", np.abs(qr), np.abs(kr[:, 0])) * rel
    top2 = np.sort(s, axis=-1)[..., -2:]
    margin = top2[..., 1] - top2[..., 0]
    # each score moves by at most its bound, so a margin above twice the bound
    # keeps the arg max, and 10 more makes the runner-up's weight < e^-10
    assert (margin > 2 * bound.max(-1) + 10).all(), "inputs must keep the arg max unambiguous"
    assert_bf16_close(o, O, "O (one key per row)")
    lerr = np.abs(f64(lse) - L)
    lbound = bound.max(-1) + np.abs(L) * 2.0 ** -23 + 1e-3   # plus the fp32 resolution of LSE itself
    assert (lerr <= lbound).all(), f"LSE error {lerr.max():.3e} above the rounding bound"
    ref = bwd_refs(lambda o_: oracle.attention_backward(fq, fk, fv, fdo, o=o_, **kw), o_ref)
    for name, gg, r in zip(("dQ", "dK", "dV"), (dq, dk, dv), ref):
        assert torch.isfinite(gg.float()).all(), name
        assert_bf16_close(gg, r, f"{name} (|q|, |k| ~ 1e3)")
