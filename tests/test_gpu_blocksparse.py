"""GPU parity of block-sparse attention (forward and backward) against the fp64
oracle with the same block mask, through the C ABI."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import (announce, assert_bf16_close, assert_lse_close, bwd_refs, device_inputs, f64, given_lse, given_o,
                      need_gpu)
from paper_2609_13612_amd import api, blockmask, inputs

pytestmark = pytest.mark.gpu


def _mask(S, density, seed, empty_rows=()):
    active = inputs.random_blocks(blockmask.num_blocks(S), density, seed=seed, empty_rows=empty_rows)
    return blockmask.block_mask_from_dense(torch.from_numpy(active), S, device="cuda")


def _fwd(dev, bm, rope, mask, window, slopes):
    return api.attnfuse_fwd_blocksparse(dev["q"], dev["k"], dev["v"], bm, rope=rope, mask=mask, window=window,
                                        alibi_slopes=slopes)


def _ref_fwd(cpu, bm, rope, mask, window, slopes):
    return oracle.attention_forward(f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), rope=rope, mask=mask,
                                    window=window, alibi_slopes=None if slopes is None else f64(slopes),
                                    block_mask=bm.as_oracle())


def _ref_bwd(cpu, bm, rope, mask, window, slopes, o_ref):
    """Oracle gradients for a backward handed ``o_ref``, the (oracle-made)
    forward output: dQ's row term from it, dK's and dV's by definition."""
    return bwd_refs(lambda o: oracle.attention_backward(
        f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), f64(cpu["do"]), rope=rope, mask=mask, window=window,
        alibi_slopes=None if slopes is None else f64(slopes), block_mask=bm.as_oracle(), o=o), o_ref)


def _bwd_given_o(cpu, dev, bm, rope, mask, window, slopes):
    """The block-sparse backward handed the oracle's forward output (O rounded
    to bf16, and its LSE), and the oracle's gradients given that O."""
    O, L = _ref_fwd(cpu, bm, rope, mask, window, slopes)
    o_ref, o_dev = given_o(O)
    grads = api.attnfuse_bwd_blocksparse(dev["q"], dev["k"], dev["v"], o_dev, dev["do"], given_lse(L), bm, rope=rope,
                                         mask=mask, window=window, alibi_slopes=slopes)
    torch.cuda.synchronize()
    return grads, _ref_bwd(cpu, bm, rope, mask, window, slopes, o_ref)


VARIANTS = list(itertools.product(["none", "neox", "interleaved"], ["none", "causal", "sliding_window"],
                                  [False, True], [64, 128]))


@pytest.mark.parametrize("rope,mask,alibi,D", VARIANTS, ids=lambda x: str(x))
def test_blocksparse_fwd_bwd_variants(rope, mask, alibi, D):
    """A random 35% block mask with one empty block row over S = 600 (ten
    blocks, the last one ragged), GQA group of two: every elementwise variant
    combined with the block mask, forward and backward."""
    need_gpu()
    B, H, Hkv, S = 1, 4, 2, 600
    window = 150 if mask == "sliding_window" else None
    announce(f"blocksparse rope={rope} mask={mask} alibi={alibi} D={D} S={S}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=31, with_do=True)
    bm = _mask(S, 0.35, seed=5, empty_rows=(3,))
    slopes = inputs.alibi_slopes(H).cuda() if alibi else None
    o, lse = _fwd(dev, bm, rope, mask, window, slopes)
    torch.cuda.synchronize()
    O, L = _ref_fwd(cpu, bm, rope, mask, window, slopes)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")
    assert torch.all(o[:, :, 3 * 64:4 * 64] == 0) and torch.all(torch.isneginf(lse[:, :, 3 * 64:4 * 64]))
    grads, ref = _bwd_given_o(cpu, dev, bm, rope, mask, window, slopes)
    for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
        assert_bf16_close(g, r, name)


@pytest.mark.parametrize("H,Hkv", [(2, 2), (8, 2), (16, 2), (8, 1)], ids=lambda x: str(x))
def test_blocksparse_group_sizes(H, Hkv):
    """GQA groups of 1, 4, 8 and 8 query heads: the forward's workgroup takes
    one query block with four, one and one key groups (its partial states
    merged when several); the dQ pass's list is the union of four, one or half
    a query block's rows."""
    need_gpu()
    B, S, D = 2, 1000, 128
    announce(f"blocksparse group H={H} Hkv={Hkv}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=32, with_do=True)
    bm = _mask(S, 0.25, seed=6)
    o, lse = _fwd(dev, bm, "neox", "causal", None, None)
    torch.cuda.synchronize()
    O, L = _ref_fwd(cpu, bm, "neox", "causal", None, None)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")
    grads, ref = _bwd_given_o(cpu, dev, bm, "neox", "causal", None, None)
    for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
        assert_bf16_close(g, r, name)


@pytest.mark.parametrize("S,mask,rope", [(600, "causal", "neox"), (333, "none", "none"),
                                         (1000, "sliding_window", "interleaved")], ids=lambda x: str(x))
def test_blocksparse_all_active_matches_dense_bitwise(S, mask, rope):
    """With every block active the tile lists equal the dense ranges, visited in
    the same order (four query heads per K/V head, so the forward runs one key
    group): the results equal the dense kernels' bit for bit."""
    need_gpu()
    B, H, Hkv, D = 1, 8, 2, 128
    window = 200 if mask == "sliding_window" else None
    announce(f"blocksparse all-active vs dense S={S} mask={mask}")
    _, dev = device_inputs(B, H, Hkv, S, D, seed=33, with_do=True)
    nb = blockmask.num_blocks(S)
    bm = blockmask.block_mask_from_dense(torch.ones(nb, nb, dtype=torch.bool), S, device="cuda")
    o, lse = _fwd(dev, bm, rope, mask, window, None)
    o2, lse2 = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=rope, mask=mask, window=window)
    g = api.attnfuse_bwd_blocksparse(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, bm, rope=rope, mask=mask,
                                     window=window)
    g2 = api.attnfuse_bwd(dev["q"], dev["k"], dev["v"], o2, dev["do"], lse2, rope=rope, mask=mask, window=window)
    torch.cuda.synchronize()
    assert torch.equal(o, o2) and torch.equal(lse, lse2)
    for a, b in zip(g, g2):
        assert torch.equal(a, b)


def test_blocksparse_empty_and_tiny():
    """No active block: O = 0, LSE = -inf, zero gradients.  S = 1 and S = 65
    (a one-position tail block) against the oracle."""
    need_gpu()
    announce("blocksparse empty mask")
    B, H, Hkv, S, D = 1, 4, 2, 200, 64
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=34, with_do=True)
    nb = blockmask.num_blocks(S)
    bm = blockmask.block_mask_from_dense(torch.zeros(nb, nb, dtype=torch.bool), S, device="cuda")
    o, lse = _fwd(dev, bm, "neox", "none", None, None)
    grads = api.attnfuse_bwd_blocksparse(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, bm, rope="neox",
                                         mask="none")
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(torch.isneginf(lse))
    for t in grads:
        assert torch.all(t == 0)
    for S in (1, 65):
        announce(f"blocksparse tiny S={S}")
        cpu, dev = device_inputs(1, 2, 1, S, 128, seed=35, with_do=True)
        nb = blockmask.num_blocks(S)
        active = np.ones((nb, nb), dtype=bool)
        active[-1, 0] = False
        bm = blockmask.block_mask_from_dense(torch.from_numpy(active), S, device="cuda")
        o, lse = _fwd(dev, bm, "neox", "causal", None, None)
        torch.cuda.synchronize()
        O, L = _ref_fwd(cpu, bm, "neox", "causal", None, None)
        assert_bf16_close(o, O, f"O S={S}")
        assert_lse_close(lse, L, f"LSE S={S}")
        grads, ref = _bwd_given_o(cpu, dev, bm, "neox", "causal", None, None)
        for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
            assert_bf16_close(g, r, f"{name} S={S}")


def test_blocksparse_bigbird_full_size():
    """The BigBird-like mask at N = 4096 over GPT-2-small heads (B 4, H 12,
    D 64) in the benchmark's configuration: forward rows sampled across every
    (batch, head) pair and the full backward of head (0, 0) against the oracle."""
    need_gpu()
    B, H, Hkv, S, D = 4, 12, 12, 4096, 64
    announce("blocksparse bigbird full size")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=36, with_do=True)
    active = inputs.bigbird_blocks(blockmask.num_blocks(S), seed=0)
    bm = blockmask.block_mask_from_dense(torch.from_numpy(active), S, device="cuda")
    o, lse = _fwd(dev, bm, "none", "none", None, None)
    dq, dk, dv = api.attnfuse_bwd_blocksparse(dev["q"], dev["k"], dev["v"], o, dev["do"], lse, bm, rope="none",
                                              mask="none")
    torch.cuda.synchronize()
    rng = np.random.default_rng(0)
    for b in range(B):
        for h in range(H):
            rows = np.unique(np.concatenate([[0, 63, 64, S - 1], rng.integers(0, S, 12)]))
            O, L = oracle.attention_forward_rows(f64(cpu["q"][b, h]), f64(cpu["k"][b, h]), f64(cpu["v"][b, h]),
                                                 rows, mask="none", block_mask=bm.as_oracle())
            assert_bf16_close(f64(o[b, h])[rows], O, f"O b={b} h={h}")
            assert_lse_close(f64(lse[b, h])[rows], L, f"LSE b={b} h={h}")
    # end to end (the backward on the GPU forward's output) against the exact
    # gradients of head (0, 0)
    ref = oracle.attention_backward(f64(cpu["q"][:1, :1]), f64(cpu["k"][:1, :1]), f64(cpu["v"][:1, :1]),
                                    f64(cpu["do"][:1, :1]), mask="none", block_mask=bm.as_oracle())
    assert_bf16_close(f64(dq[:1, :1]), ref[0], "dQ (0, 0) definitional")
    assert_bf16_close(f64(dk[:1, :1]), ref[1], "dK (0, 0) definitional")
    assert_bf16_close(f64(dv[:1, :1]), ref[2], "dV (0, 0) definitional")
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()


def test_blocksparse_reports_errors():
    need_gpu()
    _, dev = device_inputs(1, 2, 2, 128, 64, seed=0)
    bm = _mask(256, 0.5, seed=0)
    with pytest.raises(ValueError):
        _fwd(dev, bm, "none", "none", None, None)              # mask built for another S
    bm = _mask(128, 0.5, seed=0)
    with pytest.raises(api.AttnFuseError) as e:
        api.attnfuse_fwd_blocksparse(dev["q"].float(), dev["k"].float(), dev["v"].float(), bm)
    assert e.value.code == -2                                   # bf16 kernels only


def test_blocksparse_noncanonical_lists():
    """Rows in any order with duplicates, and entries outside [0, nb), describe
    the same mask as the canonical lists: duplicates count once and invalid
    entries are ignored (forward through the general list builder, backward
    through the union builder)."""
    need_gpu()
    B, H, Hkv, S, D = 1, 4, 2, 700, 64
    announce("blocksparse non-canonical lists")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=37, with_do=True)
    nb = blockmask.num_blocks(S)
    active = inputs.random_blocks(nb, 0.4, seed=9, empty_rows=(2,))
    rng = np.random.default_rng(3)

    def scrambled(mat):
        ptr, idx = [0], []
        for r in range(mat.shape[0]):
            row = list(np.flatnonzero(mat[r]))
            row += list(rng.choice(row, size=min(2, len(row)), replace=False)) if row else []   # duplicates
            row += [-1, nb + 3] if r % 3 == 0 else []                                       # invalid entries
            rng.shuffle(row)
            idx += row
            ptr.append(len(idx))
        return (torch.tensor(ptr, dtype=torch.int32, device="cuda"),
                torch.tensor(idx, dtype=torch.int32, device="cuda"))

    q_ptr, k_idx = scrambled(active)
    k_ptr, q_idx = scrambled(active.T)
    bm = blockmask.BlockMask(S, torch.from_numpy(active).cuda(), q_ptr, k_idx, k_ptr, q_idx)
    o, lse = _fwd(dev, bm, "neox", "causal", None, None)
    torch.cuda.synchronize()
    O, L = _ref_fwd(cpu, bm, "neox", "causal", None, None)
    assert_bf16_close(o, O, "O")
    assert_lse_close(lse, L, "LSE")
    grads, ref = _bwd_given_o(cpu, dev, bm, "neox", "causal", None, None)
    for name, g, r in zip(("dQ", "dK", "dV"), grads, ref):
        assert_bf16_close(g, r, name)
