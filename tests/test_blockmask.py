"""Host-side block-mask construction (CPU): the compressed lists the kernels
walk describe exactly the bool block matrix, in both orientations."""
import numpy as np
import pytest
import torch

from paper_2609_13612_amd import blockmask, inputs


def _decompress(ptr, idx, nb):
    ptr = ptr.cpu().numpy()
    idx = idx.cpu().numpy()
    out = np.zeros((nb, nb), dtype=bool)
    for r in range(nb):
        row = idx[ptr[r]:ptr[r + 1]]
        assert np.all(np.diff(row) > 0), "entries ascending, no duplicates"
        out[r, row] = True
    return out


@pytest.mark.parametrize("S,density,seed", [(1, 1.0, 0), (64, 0.5, 1), (65, 0.5, 2), (600, 0.3, 3),
                                            (4096, 0.1, 4), (64 * 2048, 0.001, 5)])
def test_csr_and_csc_describe_the_matrix(S, density, seed):
    nb = blockmask.num_blocks(S)
    active = inputs.random_blocks(nb, density, seed=seed)
    m = blockmask.block_mask_from_dense(torch.from_numpy(active), S)
    assert m.nb == nb
    for t in (m.q_ptr, m.k_idx, m.k_ptr, m.q_idx):
        assert t.dtype == torch.int32 and t.is_contiguous()
    assert m.q_ptr[0] == 0 and m.q_ptr[-1] == active.sum() == m.k_ptr[-1]
    assert np.array_equal(_decompress(m.q_ptr, m.k_idx, nb), active)
    assert np.array_equal(_decompress(m.k_ptr, m.q_idx, nb), active.T)
    assert m.density() == pytest.approx(active.mean())
    bs, act = m.as_oracle()
    assert bs == 64 and np.array_equal(act, active)


def test_create_block_mask_vectorised_and_scalar_predicates():
    S = 1000
    nb = blockmask.num_blocks(S)
    band = blockmask.create_block_mask(lambda i, j: abs(i - j) <= 1, S)     # works on arrays
    ref = np.abs(np.arange(nb)[:, None] - np.arange(nb)[None, :]) <= 1
    assert np.array_equal(band.active.numpy(), ref)

    def scalar_only(i, j):
        if not isinstance(i, (int, np.integer)):
            raise TypeError("scalars only")
        return (i + j) % 3 == 0
    m = blockmask.create_block_mask(scalar_only, S)
    ref = (np.arange(nb)[:, None] + np.arange(nb)[None, :]) % 3 == 0
    assert np.array_equal(m.active.numpy(), ref)
    const = blockmask.create_block_mask(lambda i, j: True, S)                # a scalar broadcasts
    assert const.active.all()


def test_from_csr_round_trip_and_validation():
    S = 300
    nb = blockmask.num_blocks(S)
    active = inputs.random_blocks(nb, 0.4, seed=7, empty_rows=(2,))
    m = blockmask.block_mask_from_dense(torch.from_numpy(active), S)
    again = blockmask.block_mask_from_csr(m.q_ptr, m.k_idx, S)
    assert np.array_equal(again.active.numpy(), active)
    with pytest.raises(ValueError):
        blockmask.block_mask_from_csr([0, 1, 1, 1, 1], [7], S)            # index out of range
    with pytest.raises(ValueError):
        blockmask.block_mask_from_csr([0, 2, 1, 1, 1], [0, 1], S)         # decreasing offsets
    with pytest.raises(ValueError):
        blockmask.block_mask_from_csr([1, 1, 1, 1, 1], [0], S)            # does not start at 0
    with pytest.raises(ValueError):
        blockmask.block_mask_from_csr([0, 0, 0], [], S)                   # wrong length


def test_limits():
    with pytest.raises(ValueError):
        blockmask.block_mask_from_dense(torch.ones(2049, 2049, dtype=torch.bool), 64 * 2048 + 1)
    with pytest.raises(ValueError):
        blockmask.block_mask_from_dense(torch.ones(3, 3, dtype=torch.bool), 64 * 4)


def test_bigbird_pattern_parts():
    nb = 64
    a = inputs.bigbird_blocks(nb, window=3, n_global=1, n_random=1, seed=0)
    i = np.arange(nb)
    assert np.all(a[np.abs(i[:, None] - i[None, :]) <= 1])          # the band
    assert a[0].all() and a[:, 0].all()                              # the global block
    # one random block per row beyond band and global (none free in row 0)
    band_global = (np.abs(i[:, None] - i[None, :]) <= 1) | (i[:, None] == 0) | (i[None, :] == 0)
    extra = (a & ~band_global).sum(axis=1)
    assert extra[0] == 0 and np.all(extra[1:] == 1)
    assert np.array_equal(a, inputs.bigbird_blocks(nb, seed=0))     # seeded
    assert 0.05 < a.mean() < 0.12
