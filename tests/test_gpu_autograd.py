"""The torch.autograd wrappers (paper_2609_13612_amd.autograd) through the C ABI:
outputs and gradients are exactly those of the direct entry points, and they
match the oracle."""
import torch

import oracle
from gpu_util import announce, assert_bf16_close, device_inputs, f64, need_gpu
from paper_2609_13612_amd import api, autograd, blockmask, inputs

import pytest

pytestmark = pytest.mark.gpu


def _leaves(dev):
    return [dev[n].clone().requires_grad_() for n in ("q", "k", "v")]


def test_autograd_attention_matches_abi_and_oracle():
    need_gpu()
    announce("autograd attention")
    B, H, Hkv, S, D = 1, 8, 2, 300, 128
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=81, with_do=True)
    slopes = inputs.alibi_slopes(H).cuda()
    kw = dict(rope="neox", theta=500000.0, mask="sliding_window", window=120, alibi_slopes=slopes)
    q, k, v = _leaves(dev)
    o = autograd.attention(q, k, v, **kw)
    o.backward(dev["do"])
    o2, lse2 = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], **kw)
    g2 = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o2, dev["do"], lse2, **kw)
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), o2)
    for t, g in zip((q, k, v), g2):
        assert torch.equal(t.grad, g)
    # end to end: the gradients of the exact function (no O given to the oracle)
    okw = dict(kw, alibi_slopes=f64(slopes))
    ref = oracle.attention_backward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), f64(cpu["do"]), **okw)
    for name, t, r in zip(("dQ", "dK", "dV"), (q, k, v), ref):
        assert_bf16_close(t.grad, r, f"{name} definitional")


def test_autograd_loss_of_output():
    """A scalar loss of O: the gradient reaching O is 2 O (in fp32, then bf16),
    and the leaves' gradients equal attnfuse_bwd on that gradient."""
    need_gpu()
    announce("autograd loss")
    B, H, Hkv, S, D = 2, 4, 4, 200, 64
    _, dev = device_inputs(B, H, Hkv, S, D, seed=82)
    q, k, v = _leaves(dev)
    o, lse = autograd.attention(q, k, v, rope="interleaved", mask="causal", return_lse=True)
    assert not lse.requires_grad
    loss = (o.float() ** 2).sum()
    loss.backward()
    do = (2 * o.detach().float()).to(torch.bfloat16)
    g2 = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o.detach(), do, lse, rope="interleaved", mask="causal")
    torch.cuda.synchronize()
    for t, g in zip((q, k, v), g2):
        assert torch.equal(t.grad, g)


def test_autograd_blocksparse():
    need_gpu()
    announce("autograd block-sparse")
    B, H, Hkv, S, D = 1, 4, 4, 1024, 64
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=83, with_do=True)
    bm = blockmask.block_mask_from_dense(torch.from_numpy(inputs.bigbird_blocks(S // 64, seed=2)), S, device="cuda")
    q, k, v = _leaves(dev)
    o = autograd.blocksparse_attention(q, k, v, bm, rope="neox")
    o.backward(dev["do"])
    o2, lse2 = api.attnfuse_fwd_blocksparse(dev["q"], dev["k"], dev["v"], bm, rope="neox")
    g2 = api.attnfuse_bwd_blocksparse(dev["q"], dev["k"], dev["v"], o2, dev["do"], lse2, bm, rope="neox")
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), o2)
    for t, g in zip((q, k, v), g2):
        assert torch.equal(t.grad, g)


@pytest.mark.parametrize("norm", ["softmax", "relu"])
def test_autograd_bias_norm(norm):
    need_gpu()
    announce(f"autograd bias norm={norm}")
    B, H, Hkv, S, D = 2, 4, 2, 160, 128
    _, dev = device_inputs(B, H, Hkv, S, D, seed=84, with_do=True)
    g = torch.Generator("cpu").manual_seed(84)
    bias = torch.randn(B, 1, S, S, generator=g, dtype=torch.float32).cuda()
    scale = D ** -0.5 / (S if norm == "relu" else 1)
    kw = dict(bias=bias / (S if norm == "relu" else 1), norm=norm, rope="neox", mask="causal", scale=scale)
    q, k, v = _leaves(dev)
    o = autograd.attention_bias_norm(q, k, v, **kw)
    o.backward(dev["do"])
    o2, lse2 = api.attnfuse_fwd_bias_norm(dev["q"], dev["k"], dev["v"], **kw)
    g2 = api.attnfuse_bwd_bias_norm(dev["q"], dev["k"], dev["v"], o2, dev["do"], lse2, **kw)
    torch.cuda.synchronize()
    assert torch.equal(o.detach(), o2)
    for t, gr in zip((q, k, v), g2):
        assert torch.equal(t.grad, gr)
