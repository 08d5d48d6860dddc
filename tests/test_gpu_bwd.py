"""GPU parity of the three-kernel backward against the fp64 oracle (through the C ABI)."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, assert_bf16_close, assert_fp32_close, device_inputs, f64, need_gpu
from paper_2609_13612_amd import api, inputs
from paper_2609_13612_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def _run(cpu, dev, B, H, Hkv, S, D, rope, theta, mask, window, alibi):
    slopes = inputs.alibi_slopes(H).cuda() if alibi else None
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=rope, theta=theta, mask=mask, window=window,
                              alibi_slopes=slopes)
    dq, dk, dv = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, rope=rope, theta=theta,
                                  mask=mask, window=window, alibi_slopes=slopes)
    torch.cuda.synchronize()
    ref = oracle.attention_backward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), f64(cpu["do"]), rope=rope,
                                    theta=theta, mask=mask, window=window,
                                    alibi_slopes=None if slopes is None else f64(slopes), o=f64(o))
    return (dq, dk, dv), ref


VARIANTS = list(itertools.product(["none", "neox", "interleaved"], ["none", "causal", "sliding_window"],
                                  [False, True], [64, 128]))


@pytest.mark.parametrize("rope,mask,alibi,D", VARIANTS, ids=lambda x: str(x))
def test_bwd_variants(rope, mask, alibi, D):
    need_gpu()
    B, H, Hkv, S = 1, 4, 2, 257
    window = 100 if mask == "sliding_window" else None
    announce(f"bwd rope={rope} mask={mask} alibi={alibi} D={D} S={S}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=11, with_do=True)
    got, ref = _run(cpu, dev, B, H, Hkv, S, D, rope, 10000.0, mask, window, alibi)
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        assert_bf16_close(g, r, name)


FP32_VARIANTS = [("neox", "sliding_window", False, 128), ("interleaved", "none", True, 64),
                 ("none", "causal", True, 128), ("neox", "causal", False, 64),
                 ("interleaved", "causal", False, 128), ("none", "sliding_window", True, 64)]


@pytest.mark.parametrize("rope,mask,alibi,D", FP32_VARIANTS, ids=lambda x: str(x))
def test_bwd_fp32_variants(rope, mask, alibi, D):
    """The fp32 debug backward against the fp64 oracle at the fp32 bound (1e-4),
    with a ragged S (two 64-row blocks and a tail) and a GQA group of two."""
    need_gpu()
    B, H, Hkv, S = 1, 4, 2, 130
    window = 50 if mask == "sliding_window" else None
    announce(f"bwd fp32 rope={rope} mask={mask} alibi={alibi} D={D} S={S}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, dtype="fp32", seed=13, with_do=True)
    got, ref = _run(cpu, dev, B, H, Hkv, S, D, rope, 10000.0, mask, window, alibi)
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        assert_fp32_close(g, r, name + " fp32")


EDGE = [
    (1, 1, 1, 1, 64, "neox", "causal", None),
    (1, 2, 1, 3, 128, "neox", "causal", None),
    (1, 2, 2, 64, 64, "interleaved", "none", None),
    (1, 2, 2, 129, 128, "neox", "causal", None),
    (2, 8, 2, 190, 128, "neox", "causal", None),
    (1, 2, 2, 300, 64, "neox", "sliding_window", 1),
    (1, 2, 2, 300, 128, "neox", "sliding_window", 130),
]


@pytest.mark.parametrize("B,H,Hkv,S,D,rope,mask,window", EDGE, ids=lambda x: str(x))
def test_bwd_edges(B, H, Hkv, S, D, rope, mask, window):
    need_gpu()
    announce(f"bwd edge B={B} H={H} Hkv={Hkv} S={S} D={D} rope={rope} mask={mask} W={window}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=12, with_do=True)
    got, ref = _run(cpu, dev, B, H, Hkv, S, D, rope, 10000.0, mask, window, False)
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        assert_bf16_close(g, r, name)


def test_bwd_llama3_full_size_one_group():
    """Full Llama-3-8B shape in the benchmark's launch configuration; the oracle
    recomputes the first K/V head's GQA group (4 query heads) exactly."""
    need_gpu()
    w = WORKLOADS["llama3_8b_b1h32kv8s8192d128"]
    announce("bwd full size llama3 (group 0)")
    cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, seed=0, with_do=True)
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=w.rope, theta=w.theta, mask=w.mask)
    dq, dk, dv = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, rope=w.rope, theta=w.theta,
                                  mask=w.mask)
    torch.cuda.synchronize()
    G = w.H // w.Hkv
    sl = slice(0, G)
    ref = oracle.attention_backward(f64(cpu["q"][:, sl]), f64(cpu["k"][:, :1]), f64(cpu["v"][:, :1]),
                                    f64(cpu["do"][:, sl]), rope=w.rope, theta=w.theta, mask=w.mask,
                                    o=f64(o[:, sl]))
    assert_bf16_close(f64(dq[:, sl]), ref[0], "dQ group 0")
    assert_bf16_close(f64(dk[:, :1]), ref[1], "dK group 0")
    assert_bf16_close(f64(dv[:, :1]), ref[2], "dV group 0")
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()


def test_bwd_separate_path_vs_oracle():
    """Backward through rotate-then-attend (the no-RoPE backward on the rotation
    kernel's bf16 tensors, then the inverse-rotation kernel) against the oracle
    gradient of the fused function.  (Two bf16 outputs that each round
    independently may differ by a full ulp, so each path is held to the oracle
    rather than to the other.)"""
    need_gpu()
    B, H, Hkv, S, D = 1, 4, 2, 300, 128
    announce("bwd separate path vs oracle")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=13, with_do=True)
    qr, kr = api.attnfuse_rope(dev["q"], dev["k"], rope="neox")
    o2, lse2 = api.attnfuse_fwd(qr, kr, dev["v"], rope="none", mask="causal")
    dqr, dkr, dv2 = api.attnfuse_bwd(qr, kr, dev["v"], o2, dev["do"], lse2, rope="none", mask="causal")
    dq2, dk2 = api.attnfuse_rope_bwd(dqr, dkr, rope="neox")
    torch.cuda.synchronize()
    ref = oracle.attention_backward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), f64(cpu["do"]), rope="neox",
                                    mask="causal", o=f64(o2))
    for name, g, r in zip(("dQ", "dK", "dV"), (dq2, dk2, dv2), ref):
        assert_bf16_close(g, r, f"separate path {name}")
