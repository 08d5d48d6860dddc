"""GPU parity of the additive-bias and relu-attention variants (forward and
backward) against the fp64 oracle, through the C ABI."""
import itertools

import pytest
import torch

import oracle
from gpu_util import (announce, assert_bf16_close, assert_lse_close, bwd_refs, device_inputs, f64, given_lse, given_o,
                      need_gpu)
from paper_2609_13612_amd import api

pytestmark = pytest.mark.gpu


def _bias(kind, B, H, S, seed):
    """fp32 CPU bias: 'full' [B, H, S, S] N(0, 1.5^2); 'keypad' [B, 1, 1, S] with
    the last keys of each sequence at -inf (a key-padding mask as a bias)."""
    g = torch.Generator("cpu").manual_seed(seed)
    if kind == "full":
        return 1.5 * torch.randn(B, H, S, S, generator=g, dtype=torch.float32)
    pad = torch.zeros(B, 1, 1, S, dtype=torch.float32)
    for b in range(B):
        pad[b, ..., S - 7 * (b + 1):] = -float("inf")
    return pad


def _run(B, H, Hkv, S, D, *, rope, mask, window, bias_kind, norm, seed):
    """Relu attention runs in its published form relu(s / L) with L = S, the
    sequence length: the 1/L is folded into the scale and the bias, so outputs
    stay O(1) like the softmax's (unnormalised sums over hundreds of keys would
    be dominated by bf16 storage rounding)."""
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=seed, with_do=True)
    bias = None if bias_kind is None else _bias(bias_kind, B, H, S, seed)
    scale = D ** -0.5
    if norm == "relu":
        scale /= S
        bias = None if bias is None else bias / S
    dbias = None if bias is None else bias.cuda()
    o, lse = api.attnfuse_fwd_bias_norm(dev["q"], dev["k"], dev["v"], bias=dbias, norm=norm, rope=rope, mask=mask,
                                        window=window, scale=scale)
    ob = None if bias is None else bias.to(torch.float64).numpy()
    kw = dict(rope=rope, mask=mask, window=window, bias=ob, norm=norm, scale=scale)
    O, L = oracle.attention_forward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), **kw)
    # the backward is handed the oracle's forward output (rounded to bf16)
    o_ref, o_dev = given_o(O)
    grads = api.attnfuse_bwd_bias_norm(dev["q"], dev["k"], dev["v"], o_dev, dev["do"],
                                       None if L is None else given_lse(L), bias=dbias, norm=norm, rope=rope,
                                       mask=mask, window=window, scale=scale)
    torch.cuda.synchronize()
    # the relu gate s > 0 is a decision: both sides take it on fp16 operands
    # (the kernels' MFMA operand type in the backward)
    ref = bwd_refs(lambda o_: oracle.attention_backward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), f64(cpu["do"]),
                                                        relu_gate="fp16" if norm == "relu" else "exact", o=o_, **kw),
                   o_ref)
    return (o, lse, grads), (O, L, ref)


VARIANTS = list(itertools.product(["none", "neox", "interleaved"], ["none", "causal", "sliding_window"],
                                  [("full", "softmax"), (None, "relu"), ("full", "relu")], [64, 128]))


@pytest.mark.parametrize("rope,mask,ext,D", VARIANTS, ids=lambda x: str(x))
def test_bias_relu_variants(rope, mask, ext, D):
    """S = 300 (four 64-key tiles and a ragged tail), GQA group of two, every
    RoPE kind and mask with a dense bias, relu attention, or both."""
    need_gpu()
    bias_kind, norm = ext
    window = 90 if mask == "sliding_window" else None
    announce(f"bias/relu rope={rope} mask={mask} bias={bias_kind} norm={norm} D={D}")
    (o, lse, grads), (O, L, ref) = _run(1, 4, 2, 300, D, rope=rope, mask=mask, window=window, bias_kind=bias_kind,
                                        norm=norm, seed=51)
    assert_bf16_close(o, O, "O")
    if norm == "softmax":
        assert_lse_close(lse, L, "LSE")
    else:
        assert lse is None
    for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
        assert_bf16_close(g, r, name)


@pytest.mark.parametrize("norm", ["softmax", "relu"])
def test_key_padding_bias_broadcast(norm):
    """A [B, 1, 1, S] bias broadcast over heads and queries (strides 0) with
    -inf on padded keys; batch 2 with different padding, NeoX RoPE, no
    elementwise mask."""
    need_gpu()
    announce(f"key-padding bias norm={norm}")
    (o, lse, grads), (O, L, ref) = _run(2, 8, 2, 260, 128, rope="neox", mask="none", window=None, bias_kind="keypad",
                                        norm=norm, seed=52)
    assert_bf16_close(o, O, "O")
    if norm == "softmax":
        assert_lse_close(lse, L, "LSE")
    for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
        assert_bf16_close(g, r, name)


def test_plain_softmax_equals_attnfuse_fwd():
    """bias = None with the softmax is the plain forward and backward, bit for bit."""
    need_gpu()
    announce("bias_norm without bias vs attnfuse_fwd")
    _, dev = device_inputs(1, 8, 2, 500, 128, seed=53, with_do=True)
    o1, l1 = api.attnfuse_fwd_bias_norm(dev["q"], dev["k"], dev["v"], rope="neox", mask="causal")
    o2, l2 = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope="neox", mask="causal")
    g1 = api.attnfuse_bwd_bias_norm(dev["q"], dev["k"], dev["v"], o1, dev["do"], l1, rope="neox", mask="causal")
    g2 = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o2, dev["do"], l2, rope="neox", mask="causal")
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    for a, b in zip(g1, g2):
        assert torch.equal(a, b)


def test_bias_relu_larger():
    """S = 1024 with a dense bias under relu attention, B 2, H 8 / H_kv 2, D 128,
    sliding window 300, interleaved RoPE."""
    need_gpu()
    announce("bias+relu S=1024")
    (o, _, grads), (O, _, ref) = _run(2, 8, 2, 1024, 128, rope="interleaved", mask="sliding_window", window=300,
                                      bias_kind="full", norm="relu", seed=54)
    assert_bf16_close(o, O, "O")
    for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
        assert_bf16_close(g, r, name)


def test_bias_relu_reports_errors():
    need_gpu()
    _, dev = device_inputs(1, 2, 2, 64, 64, seed=0)
    with pytest.raises(ValueError):
        api.attnfuse_fwd_bias_norm(dev["q"], dev["k"], dev["v"], bias=torch.zeros(1, 2, 64, 64, device="cuda",
                                                                                   dtype=torch.float16))
    with pytest.raises(api.AttnFuseError) as e:
        api.attnfuse_fwd_bias_norm(dev["q"].float(), dev["k"].float(), dev["v"].float(), norm="relu")
    assert e.value.code == -2
