"""Seeded synthetic inputs shared by the HIP path's tests, the bench and the oracle checks.

This module holds none of the method's arithmetic.  It draws i.i.d. N(0, 1)
tensors from a CPU ``torch.Generator`` in a fixed order -- Q, K, V, then dO
(decode: the query, then the K and V caches) -- as fp32, and rounds them to
the storage dtype (bf16 rounds to nearest even).
Both sides of a parity check consume exactly these values: the HIP path after
a copy to the GPU, the oracle after an exact upcast to fp64.
Block-sparse patterns are bool matrices over (query block, key block), drawn
from a numpy ``Generator`` of their own seed.
"""
import numpy as np
import torch

DTYPES = {"bf16": torch.bfloat16, "fp32": torch.float32}


def make_qkv(B, H, Hkv, S, D, *, dtype="bf16", seed=0, with_do=False):
    """Dict with q [B,H,S,D], k and v [B,Hkv,S,D] (and do [B,H,S,D]) on the CPU."""
    if dtype not in DTYPES:
        raise ValueError(f"dtype must be one of {sorted(DTYPES)}")
    g = torch.Generator("cpu").manual_seed(seed)
    out = {
        "q": torch.randn(B, H, S, D, generator=g, dtype=torch.float32),
        "k": torch.randn(B, Hkv, S, D, generator=g, dtype=torch.float32),
        "v": torch.randn(B, Hkv, S, D, generator=g, dtype=torch.float32),
    }
    if with_do:
        out["do"] = torch.randn(B, H, S, D, generator=g, dtype=torch.float32)
    t = DTYPES[dtype]
    return {name: x.to(t).contiguous() for name, x in out.items()}


def make_decode(B, H, Hkv, S_kv, D, *, dtype="bf16", seed=0):
    """Dict with q [B,H,D] (one query per sequence) and the caches k, v
    [B,Hkv,S_kv,D] on the CPU, drawn in that order."""
    if dtype not in DTYPES:
        raise ValueError(f"dtype must be one of {sorted(DTYPES)}")
    g = torch.Generator("cpu").manual_seed(seed)
    out = {
        "q": torch.randn(B, H, D, generator=g, dtype=torch.float32),
        "k": torch.randn(B, Hkv, S_kv, D, generator=g, dtype=torch.float32),
        "v": torch.randn(B, Hkv, S_kv, D, generator=g, dtype=torch.float32),
    }
    t = DTYPES[dtype]
    return {name: x.to(t).contiguous() for name, x in out.items()}


def alibi_slopes(H):
    """The ALiBi workload's per-head slopes 2^(-8h/H) for h = 1..H, as fp32 [H]."""
    h = torch.arange(1, H + 1, dtype=torch.float64)
    return torch.pow(2.0, -8.0 * h / H).to(torch.float32)


def to_f64(t):
    """Exact upcast of a (CPU or GPU) tensor to an fp64 numpy array."""
    return t.detach().to("cpu", torch.float64).numpy()


def random_blocks(nb, density, *, seed=0, empty_rows=()):
    """Bool [nb, nb]: each (query block, key block) active with probability
    ``density``; the rows listed in ``empty_rows`` have no active block."""
    rng = np.random.default_rng(seed)
    active = rng.random((nb, nb)) < density
    for r in empty_rows:
        active[r] = False
    return active


def bigbird_blocks(nb, *, window=3, n_global=1, n_random=1, seed=0):
    """Bool [nb, nb] with the three parts of a BigBird-style mask: a band of
    ``window`` blocks around the diagonal, ``n_global`` global blocks (the
    first block rows see every key block and every query block sees the first
    key blocks), and ``n_random`` further key blocks per query block drawn
    uniformly from those not yet active."""
    rng = np.random.default_rng(seed)
    i = np.arange(nb)
    active = np.abs(i[:, None] - i[None, :]) <= window // 2
    active[:n_global, :] = True
    active[:, :n_global] = True
    for r in range(nb):
        free = np.flatnonzero(~active[r])
        if free.size:
            active[r, rng.choice(free, size=min(n_random, free.size), replace=False)] = True
    return active
