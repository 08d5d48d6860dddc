"""The seeded input generators every parity test, the bench and smoke() share:
the ALiBi slope recipe against its closed form, the N(0, 1) draws (shapes,
storage rounding, determinism, moments), and the block-mask patterns against
their stated structure (CPU)."""
import numpy as np
import pytest
import torch

from paper_2609_13612_amd import inputs
from paper_2609_13612_amd.workloads import SPARSE_WORKLOADS


def test_alibi_slopes_closed_form():
    # H = 8: the slopes are exactly 1/2, 1/4, ..., 1/256
    assert torch.equal(inputs.alibi_slopes(8), torch.tensor([2.0 ** -h for h in range(1, 9)]))
    # H = 16: a geometric sequence of ratio 2^-1/2 from 2^-1/2 down to exactly 2^-8
    s32 = inputs.alibi_slopes(16)
    assert s32.dtype == torch.float32 and s32.shape == (16,)
    s = s32.double()
    assert s[-1].item() == 2.0 ** -8 and s[1].item() == 0.5
    assert torch.allclose(s[1:] / s[:-1], torch.full((15,), 2.0 ** -0.5, dtype=torch.float64), rtol=1e-6)


def test_make_qkv_shapes_dtypes_and_rounding():
    c = inputs.make_qkv(2, 4, 2, 33, 64, seed=5, with_do=True)
    assert c["q"].shape == (2, 4, 33, 64) and c["do"].shape == (2, 4, 33, 64)
    assert c["k"].shape == (2, 2, 33, 64) and c["v"].shape == (2, 2, 33, 64)
    assert all(t.dtype == torch.bfloat16 and t.is_contiguous() for t in c.values())
    f = inputs.make_qkv(2, 4, 2, 33, 64, seed=5, dtype="fp32", with_do=True)
    # the bf16 tensors are the fp32 draws rounded to nearest even
    for n in ("q", "k", "v", "do"):
        assert torch.equal(c[n], f[n].to(torch.bfloat16))
    # dO is drawn after V: asking for it leaves Q, K and V unchanged
    c2 = inputs.make_qkv(2, 4, 2, 33, 64, seed=5)
    assert all(torch.equal(c[n], c2[n]) for n in ("q", "k", "v"))
    with pytest.raises(ValueError):
        inputs.make_qkv(1, 1, 1, 1, 64, dtype="fp16")


def test_make_qkv_seeded_and_standard_normal():
    a = inputs.make_qkv(1, 8, 8, 512, 128, seed=11, dtype="fp32")
    b = inputs.make_qkv(1, 8, 8, 512, 128, seed=11, dtype="fp32")
    c = inputs.make_qkv(1, 8, 8, 512, 128, seed=12, dtype="fp32")
    assert all(torch.equal(a[n], b[n]) for n in a)
    assert not torch.equal(a["q"], c["q"])
    x = torch.cat([a[n].flatten() for n in ("q", "k", "v")]).double()   # 1.5M draws
    assert abs(x.mean().item()) < 5e-3 and abs(x.std().item() - 1.0) < 5e-3
    assert abs((x ** 4).mean().item() - 3.0) < 0.05                       # normal kurtosis


def test_make_decode_order_and_shapes():
    d = inputs.make_decode(3, 8, 2, 100, 128, seed=4)
    assert d["q"].shape == (3, 8, 128) and d["k"].shape == (3, 2, 100, 128) and d["v"].shape == d["k"].shape
    g = torch.Generator("cpu").manual_seed(4)
    q = torch.randn(3, 8, 128, generator=g).to(torch.bfloat16)
    assert torch.equal(d["q"], q)


def test_random_blocks_density_and_empty_rows():
    a = inputs.random_blocks(64, 0.25, seed=3, empty_rows=(0, 17))
    assert a.dtype == bool and a.shape == (64, 64)
    assert not a[0].any() and not a[17].any()
    assert abs(a.mean() - 0.25 * 62 / 64) < 0.03
    assert np.array_equal(a, inputs.random_blocks(64, 0.25, seed=3, empty_rows=(0, 17)))


@pytest.mark.parametrize("nb,window,n_global,n_random", [(64, 3, 1, 1), (32, 5, 2, 3), (4, 3, 1, 5)])
def test_bigbird_blocks_structure(nb, window, n_global, n_random):
    a = inputs.bigbird_blocks(nb, window=window, n_global=n_global, n_random=n_random, seed=9)
    i = np.arange(nb)
    band = np.abs(i[:, None] - i[None, :]) <= window // 2
    assert a[band].all()                                   # the band around the diagonal
    assert a[:n_global].all() and a[:, :n_global].all()    # global rows and columns
    fixed = band.copy()
    fixed[:n_global] = True
    fixed[:, :n_global] = True
    extra = (a & ~fixed).sum(axis=1)
    free = (~fixed).sum(axis=1)
    # exactly n_random further blocks per row, or all that remain
    assert np.array_equal(extra, np.minimum(n_random, free))


def test_bigbird_workload_density():
    w = SPARSE_WORKLOADS["bigbird_b4h12s4096d64"]
    a = w.active()
    nb = w.S // 64
    assert a.shape == (nb, nb)
    # band 3 blocks (2 at the ends), one global row and column, one random block per row
    band = 3 * nb - 2
    fixed = band + (nb - 2) + (nb - 2)      # the global row and column outside the band
    assert a.sum() == fixed + (nb - 1)      # every non-global row gains one random block
    assert abs(a.mean() - 0.092) < 0.001
