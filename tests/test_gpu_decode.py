"""GPU parity of decode attention (attnfuse_decode) against the fp64 oracle, through the C ABI."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import announce, assert_bf16_close, assert_lse_close, f64, need_gpu
from paper_2609_13612_amd import api, inputs
from paper_2609_13612_amd.workloads import DECODE_WORKLOADS

pytestmark = pytest.mark.gpu


def _case(B, H, Hkv, S, D, seed):
    """Seeded query [B, H, D] and caches [B, Hkv, S, D] (the caches stand for
    keys already rotated at their positions)."""
    c = inputs.make_decode(B, H, Hkv, S, D, seed=seed)
    return c["q"], c["k"], c["v"]


def _run(B, H, Hkv, S, D, *, lens=None, rope="none", theta=10000.0, mask="causal", window=None, alibi=False,
         seed=0):
    q, kc, vc = _case(B, H, Hkv, S, D, seed)
    slopes = inputs.alibi_slopes(H) if alibi else None
    dev_lens = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
    o, lse = api.attnfuse_decode(q.cuda(), kc.cuda(), vc.cuda(), dev_lens, rope=rope, theta=theta, mask=mask,
                                 window=window, alibi_slopes=None if slopes is None else slopes.cuda())
    torch.cuda.synchronize()
    ref_lens = None if lens is None else [min(max(x, 0), S) for x in lens]
    live = [b for b in range(B) if ref_lens is None or ref_lens[b] >= 1]
    O = np.zeros((B, H, D))
    L = np.full((B, H), -np.inf)
    if live:
        Ol, Ll = oracle.decode_forward(f64(q)[live], f64(kc)[live], f64(vc)[live],
                                       None if ref_lens is None else [ref_lens[b] for b in live], rope=rope,
                                       theta=theta, mask=mask, window=window,
                                       alibi_slopes=None if slopes is None else f64(slopes))
        O[live], L[live] = Ol, Ll
    return o, lse, O, L


VARIANTS = list(itertools.product(["none", "neox", "interleaved"], ["causal", "sliding_window"], [False, True],
                                  [64, 128]))


@pytest.mark.parametrize("rope,mask,alibi,D", VARIANTS, ids=lambda x: str(x))
def test_decode_variants(rope, mask, alibi, D):
    """A ragged batch of two sequences (700 and 333 cached keys; neither a
    multiple of the 128-key chunk), GQA group of 4."""
    need_gpu()
    announce(f"decode rope={rope} mask={mask} alibi={alibi} D={D}")
    window = 100 if mask == "sliding_window" else None
    o, lse, O, L = _run(2, 8, 2, 700, D, lens=[700, 333], rope=rope, mask=mask, window=window, alibi=alibi, seed=21)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")


@pytest.mark.parametrize("H,Hkv", [(4, 4), (32, 8), (64, 8), (32, 1)], ids=lambda x: str(x))
def test_decode_group_sizes(H, Hkv):
    """Query heads per K/V head 1, 4, 8 and 32 (every MFMA column a distinct head)."""
    need_gpu()
    announce(f"decode group H={H} Hkv={Hkv}")
    o, lse, O, L = _run(1, H, Hkv, 1500, 128, rope="neox", theta=500000.0, seed=22)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")


def test_decode_edges():
    """Cache length 1 (O = v_0), lengths above S_kv (clamped), 0 (empty: O = 0,
    LSE = -inf), and a width-1 window (O = the newest value)."""
    need_gpu()
    announce("decode edges")
    o, lse, O, L = _run(4, 8, 2, 260, 128, lens=[1, 260, 999, 0], rope="neox", seed=23)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")
    assert torch.all(o[3] == 0) and torch.all(torch.isneginf(lse[3]))
    _, kc, vc = _case(4, 8, 2, 260, 128, 23)
    assert torch.equal(o[0].cpu(), vc[0, :, 0].repeat_interleave(4, dim=0))   # bf16 v_0 exactly
    o, lse, O, L = _run(2, 4, 1, 300, 64, lens=[300, 17], mask="sliding_window", window=1, rope="interleaved",
                        seed=24)
    assert_bf16_close(o, O, "O window 1")
    assert_lse_close(lse, L, "LSE window 1")


@pytest.mark.parametrize("mask,window", [("causal", None), ("sliding_window", 12000)], ids=str)
def test_decode_many_chunks(mask, window):
    """A long cache over one K/V head: 157 chunks of 128 keys, so the merge runs
    past the 64 partials each thread loads up front (95 under the window, 71 for
    the shorter sequence)."""
    need_gpu()
    announce(f"decode many chunks mask={mask}")
    o, lse, O, L = _run(2, 4, 1, 20000, 128, lens=[20000, 9000], rope="neox", theta=500000.0, mask=mask,
                        window=window, seed=26)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")


@pytest.mark.parametrize("name", sorted(DECODE_WORKLOADS))
def test_decode_paper_geometries(name):
    """The three cache geometries of the paper's decode table at full size."""
    need_gpu()
    w = DECODE_WORKLOADS[name]
    announce(f"decode {name}")
    o, lse, O, L = _run(w.B, w.H, w.Hkv, w.S_kv, w.D, rope=w.rope, theta=w.theta, seed=25)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")


def test_decode_reports_errors():
    need_gpu()
    q, kc, vc = _case(1, 4, 2, 64, 96, 0)
    with pytest.raises(api.AttnFuseError) as e:
        api.attnfuse_decode(q.cuda(), kc.cuda(), vc.cuda())
    assert e.value.code == -2
