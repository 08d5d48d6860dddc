"""Block masks for block-sparse attention (Section 4.3 "Block-Sparse Attention").

Positions are grouped into blocks of ``BLOCK`` = 64; a mask says which (query
block, key block) pairs are active.  ``create_block_mask`` evaluates a
predicate over block coordinates once and stores the result in the two
compressed forms the kernels walk: by query block (CSR: ``q_ptr`` / ``k_idx``,
used by the forward and the dQ pass) and by key block (CSC: ``k_ptr`` /
``q_idx``, used by the dK/dV pass).  Building the lists is host-side (or torch
on the mask's device) set-up, done once per mask; no attention arithmetic
happens here.
"""
from dataclasses import dataclass

import numpy as np
import torch

BLOCK = 64
MAX_BLOCKS = 2048          # per side; S <= 64 * 2048


def num_blocks(S):
    return (S + BLOCK - 1) // BLOCK


@dataclass(frozen=True)
class BlockMask:
    """One block mask shared by every batch and head.

    ``active`` is the bool matrix [nb, nb] (on the lists' device); the four
    int32 tensors are the compressed lists, each row's / column's entries
    ascending."""
    S: int
    active: torch.Tensor
    q_ptr: torch.Tensor
    k_idx: torch.Tensor
    k_ptr: torch.Tensor
    q_idx: torch.Tensor

    @property
    def nb(self):
        return self.active.shape[0]

    @property
    def device(self):
        return self.q_ptr.device

    def density(self):
        """Fraction of the nb x nb blocks that are active."""
        return float(self.active.sum()) / float(self.nb * self.nb)

    def to(self, device):
        return BlockMask(self.S, *(t.to(device) for t in (self.active, self.q_ptr, self.k_idx, self.k_ptr,
                                                           self.q_idx)))

    def as_oracle(self):
        """The (block size, bool numpy matrix) pair the oracle takes."""
        return BLOCK, self.active.cpu().numpy().astype(bool)


def _compress(active):
    """(ptr, idx) of the rows of a bool matrix, int32, on its device."""
    counts = active.sum(dim=1, dtype=torch.int64)
    ptr = torch.zeros(active.shape[0] + 1, dtype=torch.int64, device=active.device)
    ptr[1:] = torch.cumsum(counts, 0)
    idx = active.nonzero()[:, 1]           # row-major: rows ascending, columns ascending within a row
    return ptr.to(torch.int32).contiguous(), idx.to(torch.int32).contiguous()


def block_mask_from_dense(active, S, device=None):
    """BlockMask from a bool matrix [nb, nb] with nb = ceil(S / 64)."""
    active = torch.as_tensor(active, dtype=torch.bool)
    nb = num_blocks(S)
    if S < 1 or nb > MAX_BLOCKS:
        raise ValueError(f"block-sparse attention needs 1 <= S <= {BLOCK * MAX_BLOCKS}")
    if active.shape != (nb, nb):
        raise ValueError(f"active must be [{nb}, {nb}] for S={S}")
    if device is not None:
        active = active.to(device)
    active = active.contiguous()
    q_ptr, k_idx = _compress(active)
    k_ptr, q_idx = _compress(active.t().contiguous())
    return BlockMask(S, active, q_ptr, k_idx, k_ptr, q_idx)


def create_block_mask(predicate, S, device=None):
    """Evaluate ``predicate(q_block, k_block) -> bool`` once over every pair of
    block coordinates and compress the result.  The predicate is first called
    with broadcastable integer arrays ([nb, 1] and [1, nb]); if it cannot take
    arrays it is called once per pair."""
    nb = num_blocks(S)
    qb = np.arange(nb).reshape(nb, 1)
    kb = np.arange(nb).reshape(1, nb)
    try:
        active = np.broadcast_to(np.asarray(predicate(qb, kb), dtype=bool), (nb, nb))
    except (TypeError, ValueError):
        active = np.array([[bool(predicate(i, j)) for j in range(nb)] for i in range(nb)], dtype=bool)
    return block_mask_from_dense(torch.from_numpy(np.array(active, dtype=bool)), S, device)


def block_mask_from_csr(q_ptr, k_idx, S, device=None):
    """BlockMask from a caller's compressed rows (host-checked: offsets start at
    0, never decrease and end at len(k_idx); indices lie in [0, nb))."""
    nb = num_blocks(S)
    ptr = np.asarray(torch.as_tensor(q_ptr).cpu(), dtype=np.int64)
    idx = np.asarray(torch.as_tensor(k_idx).cpu(), dtype=np.int64)
    if ptr.shape != (nb + 1,) or ptr[0] != 0 or np.any(np.diff(ptr) < 0) or ptr[-1] != idx.size:
        raise ValueError("q_ptr must be nb+1 non-decreasing offsets from 0 to len(k_idx)")
    if idx.size and (idx.min() < 0 or idx.max() >= nb):
        raise ValueError("k_idx entries must lie in [0, nb)")
    active = np.zeros((nb, nb), dtype=bool)
    rows = np.repeat(np.arange(nb), np.diff(ptr))
    active[rows, idx] = True
    return block_mask_from_dense(torch.from_numpy(active), S, device)
