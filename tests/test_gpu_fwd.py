"""GPU parity of the fused forward and the standalone rotation against the fp64 oracle.

Every call goes through the C ABI (paper_2609_13612_amd.api marshals torch
tensors into it).  Small cases span several 128-query / 64-key tiles and a
ragged tail; full-size workloads are checked on sampled rows of sampled heads
that the oracle computes one by one.
"""
import itertools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import (announce, assert_bf16_close, assert_fp32_close, assert_lse_close, bf16_round, device_inputs,
                      f64, need_gpu)
from paper_2609_13612_amd import api, inputs
from paper_2609_13612_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def _slopes(H, alibi):
    return inputs.alibi_slopes(H).cuda() if alibi else None


def _oracle_fwd(cpu, rope, theta, mask, window, slopes, scale=None):
    return oracle.attention_forward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), rope=rope, theta=theta, mask=mask,
                                    window=window, alibi_slopes=None if slopes is None else f64(slopes),
                                    scale=scale)


# ----------------------------------------------------------------------------- small, exhaustive
VARIANTS = list(itertools.product(["none", "neox", "interleaved"], ["none", "causal", "sliding_window"],
                                  [False, True], [64, 128]))


@pytest.mark.parametrize("rope,mask,alibi,D", VARIANTS, ids=lambda x: str(x))
def test_fwd_bf16_variants(rope, mask, alibi, D):
    need_gpu()
    B, H, Hkv, S = 2, 4, 2, 257
    window = 100 if mask == "sliding_window" else None
    announce(f"fwd bf16 rope={rope} mask={mask} alibi={alibi} D={D} S={S}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=1)
    slopes = _slopes(H, alibi)
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=rope, theta=10000.0, mask=mask, window=window,
                              alibi_slopes=slopes)
    torch.cuda.synchronize()
    O, L = _oracle_fwd(cpu, rope, 10000.0, mask, window, slopes)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")


EDGE = [
    # (B, H, Hkv, S, D, rope, mask, window)
    (1, 1, 1, 1, 64, "neox", "causal", None),
    (1, 1, 1, 1, 128, "interleaved", "none", None),
    (1, 2, 1, 2, 64, "neox", "causal", None),
    (1, 2, 2, 63, 128, "neox", "causal", None),
    (1, 2, 2, 64, 64, "neox", "none", None),
    (1, 2, 2, 65, 64, "neox", "causal", None),
    (1, 2, 2, 128, 128, "neox", "causal", None),
    (1, 2, 2, 129, 128, "interleaved", "causal", None),
    (2, 8, 1, 200, 128, "neox", "causal", None),          # GQA group of 8
    (1, 2, 2, 300, 64, "neox", "sliding_window", 1),       # width-1 window: O = V
    (1, 2, 2, 300, 64, "neox", "sliding_window", 64),
    (1, 2, 2, 300, 128, "neox", "sliding_window", 129),
    (1, 2, 2, 300, 64, "neox", "sliding_window", 1000),    # window >= S: causal
    (1, 2, 2, 1000, 128, "neox", "causal", None),
]


@pytest.mark.parametrize("B,H,Hkv,S,D,rope,mask,window", EDGE, ids=lambda x: str(x))
def test_fwd_bf16_edges(B, H, Hkv, S, D, rope, mask, window):
    need_gpu()
    announce(f"fwd edge B={B} H={H} Hkv={Hkv} S={S} D={D} rope={rope} mask={mask} W={window}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=2)
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=rope, mask=mask, window=window)
    torch.cuda.synchronize()
    O, L = _oracle_fwd(cpu, rope, 10000.0, mask, window, None)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")
    if mask == "sliding_window" and window == 1:
        assert torch.equal(o, dev["v"]), "width-1 window must return V exactly"


def test_fwd_tiny_workload_fp32_and_bf16():
    """The tiny workload (B1 H2 S128 D64, interleaved RoPE, causal) on both paths."""
    need_gpu()
    w = WORKLOADS["rope_causal_tiny"]
    for dtype in ("fp32", "bf16"):
        announce(f"fwd tiny workload {dtype}")
        cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, dtype=dtype, seed=0)
        o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=w.rope, theta=w.theta, mask=w.mask)
        torch.cuda.synchronize()
        O, L = _oracle_fwd(cpu, w.rope, w.theta, w.mask, None, None)
        if dtype == "fp32":
            assert_fp32_close(o, O, "O fp32")
            assert_lse_close(lse, L, "LSE fp32", tol=1e-4)
        else:
            assert_bf16_close(o, O, "O bf16")
            assert_lse_close(lse, L, "LSE bf16")
        # Causal row 0 sees only key 0: O_0 = v_0 (exactly, up to output rounding).
        assert np.allclose(f64(o)[:, :, 0], f64(cpu["v"])[:, :, 0], atol=1e-6 if dtype == "fp32" else 0)


@pytest.mark.parametrize("rope,mask,alibi", [("neox", "sliding_window", False), ("interleaved", "none", True),
                                             ("none", "causal", True), ("neox", "causal", False)])
def test_fwd_fp32_variants(rope, mask, alibi):
    need_gpu()
    B, H, Hkv, S, D = 1, 4, 2, 130, 128
    window = 50 if mask == "sliding_window" else None
    announce(f"fwd fp32 rope={rope} mask={mask} alibi={alibi}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, dtype="fp32", seed=3)
    slopes = _slopes(H, alibi)
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=rope, mask=mask, window=window, alibi_slopes=slopes)
    torch.cuda.synchronize()
    O, L = _oracle_fwd(cpu, rope, 10000.0, mask, window, slopes)
    assert_fp32_close(o, O, "O fp32")
    assert_lse_close(lse, L, "LSE fp32", tol=1e-4)


# ----------------------------------------------------------------------------- full size, sampled
def _sample_rows(S):
    rows = {0, 1, 63, 64, 127, 128, S // 2, S - 129, S - 2, S - 1}
    rows |= set(np.random.default_rng(S).integers(0, S, 6).tolist())
    return np.array(sorted(r for r in rows if 0 <= r < S))


def _check_sampled(w, cpu, o, lse, slopes, heads):
    G = w.H // w.Hkv
    rows = _sample_rows(w.S)
    og, lg = f64(o), f64(lse)
    for (b, h) in heads:
        g = h // G
        O, L = oracle.attention_forward_rows(f64(cpu["q"][b, h]), f64(cpu["k"][b, g]), f64(cpu["v"][b, g]), rows,
                                             h=h, H=w.H, rope=w.rope, theta=w.theta, mask=w.mask,
                                             window=w.window or None,
                                             alibi_slopes=None if slopes is None else f64(slopes))
        assert_bf16_close(og[b, h, rows], O, f"O[{b},{h}] sampled rows")
        assert_lse_close(lg[b, h, rows], L, f"LSE[{b},{h}] sampled rows")


@pytest.mark.parametrize("name", ["rope_causal_b8h16s2048d64", "rope_swa1024_b4h32kv8s8192d128",
                                  "alibi_causal_b4h16s4096d128", "llama3_8b_b1h32kv8s8192d128"])
def test_fwd_full_size_sampled(name):
    need_gpu()
    w = WORKLOADS[name]
    announce(f"fwd full size {name}")
    cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, seed=0)
    slopes = _slopes(w.H, w.alibi)
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=w.rope, theta=w.theta, mask=w.mask,
                              window=w.window or None, alibi_slopes=slopes)
    torch.cuda.synchronize()
    heads = [(0, 0), (w.B - 1, w.H - 1), (w.B // 2, w.H // 2 + 1)]
    _check_sampled(w, cpu, o, lse, slopes, heads)
    assert torch.isfinite(o.float()).all()


# ----------------------------------------------------------------------------- separate RoPE path
@pytest.mark.parametrize("rope", ["neox", "interleaved"])
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("D", [64, 128])
def test_rope_kernel_vs_oracle(rope, dtype, D):
    need_gpu()
    B, H, Hkv, S = 2, 6, 2, 333
    announce(f"rope kernel {rope} {dtype} D={D}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, dtype=dtype, seed=4)
    qr, kr = api.attnfuse_rope(dev["q"], dev["k"], rope=rope, theta=500000.0)
    torch.cuda.synchronize()
    pos = np.arange(S, dtype=np.float64)
    for got, src in ((qr, "q"), (kr, "k")):
        ref = oracle.rope_rotate(f64(cpu[src]), pos, 500000.0, rope)
        err = np.abs(f64(got) - ref)
        if dtype == "bf16":   # one rounding to bf16: within one bf16 ulp of the value
            assert (err <= 2.0 ** -7 * np.abs(ref) + 1e-6).all(), f"{src}: {err.max()}"
        else:
            assert err.max() <= 1e-5, f"{src}: {err.max()}"
    # inverse rotation restores the input (fp32 exactly up to rounding; bf16 within two roundings)
    dq, dk = api.attnfuse_rope_bwd(qr, kr, rope=rope, theta=500000.0)
    torch.cuda.synchronize()
    tol = 1e-5 if dtype == "fp32" else 2e-2
    assert np.abs(f64(dq) - f64(cpu["q"])).max() <= tol
    assert np.abs(f64(dk) - f64(cpu["k"])).max() <= tol


def test_rope_kernel_in_place_and_single_tensor():
    need_gpu()
    announce("rope in place")
    cpu, dev = device_inputs(1, 4, 2, 100, 128, seed=5)
    ref, _ = api.attnfuse_rope(dev["q"], None, rope="neox")
    x = dev["q"].clone()
    api.attnfuse_rope(x, None, rope="neox", out_q=x)
    torch.cuda.synchronize()
    assert torch.equal(x, ref)


@pytest.mark.parametrize("name", ["rope_causal_b8h16s2048d64", "llama3_8b_b1h32kv8s8192d128"])
def test_separate_path(name):
    """Rotate-then-attend: the rotation kernel writes Q' and K' as bf16 tensors,
    then the forward runs without RoPE.  Its oracle is exactly that: the fp64
    rotation rounded to bf16, attended without RoPE.  It must also agree with
    the fused path (which keeps the rotated operands at fp16 precision)."""
    need_gpu()
    w = WORKLOADS[name]
    announce(f"separate path {name}")
    cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, seed=0)
    o1, l1 = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=w.rope, theta=w.theta, mask=w.mask)
    qr, kr = api.attnfuse_rope(dev["q"], dev["k"], rope=w.rope, theta=w.theta)
    o2, l2 = api.attnfuse_fwd(qr, kr, dev["v"], rope="none", mask=w.mask)
    torch.cuda.synchronize()
    pos = np.arange(w.S, dtype=np.float64)
    G = w.H // w.Hkv
    rows = _sample_rows(w.S)
    for (b, h) in [(0, 0), (w.B - 1, w.H - 1)]:
        g = h // G
        qr_ref = bf16_round(oracle.rope_rotate(f64(cpu["q"][b, h]), pos, w.theta, w.rope))
        kr_ref = bf16_round(oracle.rope_rotate(f64(cpu["k"][b, g]), pos, w.theta, w.rope))
        O, L = oracle.attention_forward_rows(qr_ref, kr_ref, f64(cpu["v"][b, g]), rows, rope="none", mask=w.mask)
        assert_bf16_close(f64(o2)[b, h, rows], O, f"separate O[{b},{h}]")
        assert_lse_close(f64(l2)[b, h, rows], L, f"separate LSE[{b},{h}]")
    assert_bf16_close(o2, f64(o1), "separate vs fused O")


def test_fwd_reports_errors():
    need_gpu()
    _, dev = device_inputs(1, 2, 2, 16, 96, seed=6)
    with pytest.raises(api.AttnFuseError) as e:
        api.attnfuse_fwd(dev["q"], dev["k"], dev["v"])
    assert e.value.code == -2
    _, dev = device_inputs(1, 2, 2, 16, 64, seed=6)
    with pytest.raises(api.AttnFuseError) as e:
        api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], mask="sliding_window", window=0)
    assert e.value.code == -1
