"""Decode attention (one query per sequence over a KV cache), fp64 -- oracle, test infrastructure only.

The paper's Flash Decoding path (Section 4.2, "Flash Decoding"; evaluated in
Table ``tab:decode``) computes ordinary attention for a single query row per
(batch, query head) against a long key/value cache; splitting the cache into
chunks and merging partial (m, l, acc) triples by log-sum-exp is exact, so the
oracle is the plain definition, one query row at a time:

1. The query of sequence b sits at position p_b = len_b - 1 (the newest token,
   whose key and value are already the last entries of the cache); RoPE rotates
   it by p_b (Section 4.1).  The cache holds keys that were rotated at their own
   positions 0..len_b-1 when they were written, so they are used as given.
2. s_j = scale * <q', k_j> - slope_h * (p_b - j) (ALiBi, if slopes are given).
3. Mask: keys j < len_b only; a sliding window of W keeps p_b - W < j <= p_b;
   causal and "none" keep every cached key (all of them precede the query).
4. O = softmax(s) V and LSE = m + ln(l), natural log.

Readings: the query position is len_b - 1; the cache stores already-rotated
keys; query head h reads cache head h // (H / H_kv).
"""
import numpy as np

from .attention import MASK_CAUSAL, MASK_NONE, MASK_SLIDING_WINDOW, kv_head
from .rope import ROPE_NONE, rope_rotate


def query_position(cache_len):
    """Position of a sequence's query: its newest token, the last cache entry."""
    return cache_len - 1


def decode_visible(j, p, mask, window=None):
    """Boolean array: is cached key j visible to the query at position p."""
    j = np.asarray(j)
    if mask == MASK_SLIDING_WINDOW:
        return (j <= p) & (j > p - window)
    return j <= p


def decode_forward(q, k_cache, v_cache, cache_lens=None, *, rope=ROPE_NONE, theta=10000.0,
                   mask=MASK_CAUSAL, window=None, alibi_slopes=None, scale=None):
    """O [B, H, D] and LSE [B, H] (fp64) for q [B, H, D] against caches [B, H_kv, S_kv, D].

    ``cache_lens`` [B] gives each sequence's valid cache length (1..S_kv);
    None means every sequence uses all S_kv entries.
    """
    q = np.asarray(q, dtype=np.float64)
    k_cache = np.asarray(k_cache, dtype=np.float64)
    v_cache = np.asarray(v_cache, dtype=np.float64)
    if q.ndim != 3 or k_cache.ndim != 4 or v_cache.shape != k_cache.shape:
        raise ValueError("q must be [B, H, D], caches [B, H_kv, S_kv, D]")
    B, H, D = q.shape
    Hkv, S_kv = k_cache.shape[1], k_cache.shape[2]
    if k_cache.shape[0] != B or k_cache.shape[3] != D or H % Hkv:
        raise ValueError("cache shape does not match q")
    lens = np.full(B, S_kv) if cache_lens is None else np.asarray(cache_lens).astype(np.int64)
    if lens.shape != (B,) or lens.min() < 1 or lens.max() > S_kv:
        raise ValueError("cache_lens must be in 1..S_kv")
    if mask not in (MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW):
        raise ValueError(f"unknown mask {mask!r}")
    if mask == MASK_SLIDING_WINDOW and (window is None or window < 1):
        raise ValueError("sliding window needs window >= 1")
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    slopes = None if alibi_slopes is None else np.asarray(alibi_slopes, dtype=np.float64)

    O = np.zeros((B, H, D))
    LSE = np.empty((B, H))
    for b in range(B):
        n = int(lens[b])
        p = query_position(n)
        j = np.arange(n)
        keep = decode_visible(j, p, mask, window)
        for h in range(H):
            g = kv_head(h, H, Hkv)
            qr = rope_rotate(q[b, h][None, :], np.array([p]), theta, rope)[0]
            s = scale * (k_cache[b, g, :n] @ qr)
            if slopes is not None:
                s = s - slopes[h] * (p - j)
            s = np.where(keep, s, -np.inf)
            m = s.max()
            e = np.exp(s - m)
            l = e.sum()
            O[b, h] = (e / l) @ v_cache[b, g, :n]
            LSE[b, h] = m + np.log(l)
    return O, LSE
