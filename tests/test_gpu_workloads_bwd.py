"""End-to-end backward parity at the full sizes of the benchmark workloads
(through the C ABI): the GPU forward, then the GPU backward on its output, in
the launch configuration bench.py times, against the oracle's gradients of
the exact function on the heads (or rows) it can afford.

* RoPE + causal, B=8, H=16, S=2048, D=64: heads (0, 0) and (7, 15).
* RoPE + sliding window 1024, B=4, H=32, H_kv=8, S=8192, D=128: the first
  GQA group of batch 0 on a slice of 3072 positions; a row depends only on
  the W keys before it, so rows and keys W or more from the slice's start
  (and, for dK and dV, from its end) are exact (positions passed as offset).
* ALiBi + causal, no RoPE, B=4, H=16, S=4096, D=128: heads (0, 0) and (3, 15).

The Llama-3-8B shape is covered in test_gpu_bwd.py and the tiny workload
there too.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, assert_bf16_close, device_inputs, f64, need_gpu
from paper_2609_13612_amd import api, inputs
from paper_2609_13612_amd.workloads import WORKLOADS

pytestmark = pytest.mark.gpu


def _run(w):
    cpu, dev = device_inputs(w.B, w.H, w.Hkv, w.S, w.D, seed=0, with_do=True)
    slopes = inputs.alibi_slopes(w.H) if w.alibi else None
    kw = dict(rope=w.rope, theta=w.theta, mask=w.mask, window=w.window or None)
    ds = None if slopes is None else slopes.cuda()
    o, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], alibi_slopes=ds, **kw)
    grads = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, alibi_slopes=ds, **kw)
    torch.cuda.synchronize()
    for t in grads:
        assert torch.isfinite(t.float()).all()
    return cpu, grads, slopes, kw


@pytest.mark.parametrize("name", ["rope_causal_b8h16s2048d64", "alibi_causal_b4h16s4096d128"])
def test_bwd_full_size_heads(name):
    need_gpu()
    w = WORKLOADS[name]
    announce(f"bwd definitional full size {name}")
    cpu, (dq, dk, dv), slopes, kw = _run(w)
    G = w.H // w.Hkv
    for b, h in ((0, 0), (w.B - 1, w.H - 1)):
        g = h // G
        sl = None if slopes is None else f64(slopes)[h:h + 1]
        ref = oracle.attention_backward(f64(cpu["q"][b:b + 1, h:h + 1]), f64(cpu["k"][b:b + 1, g:g + 1]),
                                        f64(cpu["v"][b:b + 1, g:g + 1]), f64(cpu["do"][b:b + 1, h:h + 1]),
                                        alibi_slopes=sl, **kw)
        # with one query head per K/V head (these workloads), dK and dV of the
        # head's K/V head are that head's alone
        assert G == 1
        assert_bf16_close(f64(dq[b:b + 1, h:h + 1]), ref[0], f"dQ ({b}, {h}) definitional")
        assert_bf16_close(f64(dk[b:b + 1, g:g + 1]), ref[1], f"dK ({b}, {g}) definitional")
        assert_bf16_close(f64(dv[b:b + 1, g:g + 1]), ref[2], f"dV ({b}, {g}) definitional")


def test_bwd_full_size_sliding_window_slice():
    need_gpu()
    w = WORKLOADS["rope_swa1024_b4h32kv8s8192d128"]
    announce("bwd definitional full size sliding window (group 0, slice)")
    cpu, (dq, dk, dv), _, kw = _run(w)
    G, W, L = w.H // w.Hkv, w.window, 3072
    s0 = w.S // 2 - L // 2
    sl = slice(s0, s0 + L)
    args = [f64(cpu["q"][:1, :G, sl]), f64(cpu["k"][:1, :1, sl]), f64(cpu["v"][:1, :1, sl]),
            f64(cpu["do"][:1, :G, sl])]
    ref = oracle.attention_backward(*args, pos_offset=s0, **kw)
    rows = slice(W - 1, L)          # every key such a row sees lies inside the slice
    keys = slice(W - 1, L - W + 1)  # every query that sees such a key lies inside it
    assert_bf16_close(f64(dq[:1, :G, sl])[:, :, rows], ref[0][:, :, rows], "dQ group 0 slice definitional")
    assert_bf16_close(f64(dk[:1, :1, sl])[:, :, keys], ref[1][:, :, keys], "dK group 0 slice definitional")
    assert_bf16_close(f64(dv[:1, :1, sl])[:, :, keys], ref[2][:, :, keys], "dV group 0 slice definitional")
