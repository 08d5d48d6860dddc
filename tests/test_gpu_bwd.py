"""GPU parity of the backward against the fp64 oracle (through the C ABI).

Two kinds of test:

* given-O tests hand the kernels the oracle's own forward output, rounded to
  the tensor dtype as a forward stores it, and its LSE.  The bf16 dQ pass
  forms the softmax backward's row term from the O it is given, so dQ is held
  to the oracle given the same O; the dK/dV pass uses the dQ pass's own sum
  sum_j P_ij dP_ij, so dK and dV are held to the definition.  The fp32 debug
  backward forms the row term from its (fp32) O in both passes.  No GPU value
  enters the oracle.
* definitional tests run the GPU forward and then the GPU backward on its
  output, and compare with the oracle's gradients of the exact function
  (``o=None``: delta_i = sum_j P_ij dP_ij of the exact P).
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import (announce, assert_bf16_close, assert_fp32_close, bwd_refs, device_inputs, f64, given_lse,
                      given_o, need_gpu)
from paper_2609_13612_amd import api, inputs
from paper_2609_13612_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def _run_given_o(cpu, dev, rope, theta, mask, window, alibi, dtype="bf16"):
    H = cpu["q"].shape[1]
    slopes = inputs.alibi_slopes(H) if alibi else None
    kw = dict(rope=rope, theta=theta, mask=mask, window=window)
    args = [f64(cpu[n]) for n in ("q", "k", "v", "do")]
    oslopes = None if slopes is None else f64(slopes)
    O, L = oracle.attention_forward(*args[:3], alibi_slopes=oslopes, **kw)
    o_ref, o_dev = given_o(O, dtype)
    got = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o_dev, dev["do"], given_lse(L),
                           alibi_slopes=None if slopes is None else slopes.cuda(), **kw)
    torch.cuda.synchronize()
    backward = lambda o: oracle.attention_backward(*args, alibi_slopes=oslopes, o=o, **kw)
    ref = bwd_refs(backward, o_ref) if dtype == "bf16" else backward(o_ref)
    return got, ref


VARIANTS = list(itertools.product(["none", "neox", "interleaved"], ["none", "causal", "sliding_window"],
                                  [False, True], [64, 128]))


@pytest.mark.parametrize("rope,mask,alibi,D", VARIANTS, ids=lambda x: str(x))
def test_bwd_variants(rope, mask, alibi, D):
    need_gpu()
    B, H, Hkv, S = 1, 4, 2, 257
    window = 100 if mask == "sliding_window" else None
    announce(f"bwd rope={rope} mask={mask} alibi={alibi} D={D} S={S}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=11, with_do=True)
    got, ref = _run_given_o(cpu, dev, rope, 10000.0, mask, window, alibi)
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
    got, ref = _run_given_o(cpu, dev, rope, 10000.0, mask, window, alibi, dtype="fp32")
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
    got, ref = _run_given_o(cpu, dev, rope, 10000.0, mask, window, False)
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        assert_bf16_close(g, r, name)


def _end_to_end(dev, w_kw):
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], **w_kw)
    grads = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, **w_kw)
    torch.cuda.synchronize()
    return grads


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_bwd_definitional_tiny_workload(dtype):
    """The tiny parity workload (B=1, H=2, S=128, D=64, interleaved RoPE
    theta=1e4, causal, scale 1/8): GPU forward, then GPU backward on its own
    output, against the oracle's gradients of the exact function."""
    need_gpu()
    w = WORKLOADS["rope_causal_tiny"]
    announce(f"bwd definitional tiny workload {dtype}")
    cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, dtype=dtype, seed=0, with_do=True)
    kw = dict(rope=w.rope, theta=w.theta, mask=w.mask)
    got = _end_to_end(dev, kw)
    ref = oracle.attention_backward(*[f64(cpu[n]) for n in ("q", "k", "v", "do")], **kw)
    check = assert_bf16_close if dtype == "bf16" else assert_fp32_close
    for name, g, r in zip(("dQ", "dK", "dV"), got, ref):
        check(g, r, f"{name} definitional {dtype}")


def test_bwd_llama3_full_size_one_group():
    """Full Llama-3-8B shape in the benchmark's launch configuration, end to
    end (GPU forward, then GPU backward on its output); the oracle computes
    the first K/V head's GQA group (4 query heads) of the exact function."""
    need_gpu()
    w = WORKLOADS["llama3_8b_b1h32kv8s8192d128"]
    announce("bwd definitional full size llama3 (group 0)")
    cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, seed=0, with_do=True)
    dq, dk, dv = _end_to_end(dev, dict(rope=w.rope, theta=w.theta, mask=w.mask))
    G = w.H // w.Hkv
    sl = slice(0, G)
    ref = oracle.attention_backward(f64(cpu["q"][:, sl]), f64(cpu["k"][:, :1]), f64(cpu["v"][:, :1]),
                                    f64(cpu["do"][:, sl]), rope=w.rope, theta=w.theta, mask=w.mask)
    assert_bf16_close(f64(dq[:, sl]), ref[0], "dQ group 0 definitional")
    assert_bf16_close(f64(dk[:, :1]), ref[1], "dK group 0 definitional")
    assert_bf16_close(f64(dv[:, :1]), ref[2], "dV group 0 definitional")
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()


def test_bwd_separate_path_vs_oracle():
    """Backward through rotate-then-attend: the no-RoPE backward on rotated
    bf16 tensors, then the inverse-rotation kernel.  The separate path's
    rotated tensors are bf16, so its oracle is the fp64 rotation rounded to
    bf16, attention without RoPE on those values (O handed over rounded, as
    above), and the fp64 inverse rotation of the gradients."""
    need_gpu()
    B, H, Hkv, S, D = 1, 4, 2, 300, 128
    announce("bwd separate path vs oracle")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=13, with_do=True)
    pos = np.arange(S, dtype=np.float64)
    rot = lambda x: oracle.rope_rotate(f64(x), pos, 10000.0, "neox")
    qr_ref, qr_dev = given_o(rot(cpu["q"]))
    kr_ref, kr_dev = given_o(rot(cpu["k"]))
    O, L = oracle.attention_forward(qr_ref, kr_ref, f64(cpu["v"]), rope="none", mask="causal")
    o_ref, o_dev = given_o(O)
    dqr, dkr, dv2 = api.attnfuse_bwd(qr_dev, kr_dev, dev["v"], o_dev, dev["do"], given_lse(L), rope="none",
                                     mask="causal")
    dq2, dk2 = api.attnfuse_rope_bwd(dqr, dkr, rope="neox")
    torch.cuda.synchronize()
    rq, rk, rv = bwd_refs(lambda o: oracle.attention_backward(qr_ref, kr_ref, f64(cpu["v"]), f64(cpu["do"]),
                                                              rope="none", mask="causal", o=o), o_ref)
    ref = (oracle.rope_rotate(rq, pos, 10000.0, "neox", inverse=True),
           oracle.rope_rotate(rk, pos, 10000.0, "neox", inverse=True), rv)
    for name, g, r in zip(("dQ", "dK", "dV"), (dq2, dk2, dv2), ref):
        assert_bf16_close(g, r, f"separate path {name}")
