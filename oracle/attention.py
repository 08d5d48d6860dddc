"""Masked attention with RoPE, forward and backward, in fp64 -- oracle, test infrastructure only.

Plain definition with the score matrix materialised per (batch, head); see the
package docstring.  Steps, in the order the method states them:

1. RoPE on Q and K (Section 4.1): ``rope_rotate``.
2. Score: s_ij = scale * <q'_i, k'_j> (the scaled_dot_product combinator,
   Section 3.1).
3. Post-matmul modification (Section 3.1 combinators ``alibi``, ``causal``,
   ``sliding_window``, ``full``): bias_ij = -slope_h * (i - j) for ALiBi, then
   masked entries become -inf.  An optional block-sparse mask (Section 4.3,
   "Block-Sparse Attention") additionally hides every key whose (query block,
   key block) pair is inactive.
   An optional dense bias tensor (the ``additive_bias`` combinator) is added
   to the scaled score the same way.
4. Softmax over keys: m_i = max_j s_ij, l_i = sum_j exp(s_ij - m_i),
   P_ij = exp(s_ij - m_i) / l_i.  The ``relu_attention`` combinator replaces
   it with P_ij = max(s_ij, 0) (masked entries give 0), unnormalised.
5. O = P V and LSE_i = m_i + ln(l_i) (the one saved scalar per row, Section 4.4);
   relu attention has no row statistic.

Backward (FlashAttention-2 equations, split as in Section 4.4):
dV = P^T dO, dP = dO V^T, delta_i = sum_j P_ij dP_ij (= rowsum(dO o O)),
dS = P o (dP - delta), dQ' = scale dS K', dK' = scale dS^T Q', and the rotation
is undone with its transpose: dQ = R^T dQ', dK = R^T dK'.  For grouped-query
attention the gradients of a shared K/V head sum over its query heads.  Under
relu attention dS = dP o [s > 0] (the derivative of max(s, 0), taken as 0 at
s = 0) and there is no delta.  Neither the ALiBi slopes nor the bias tensor
receive a gradient.

Readings of points the paper leaves open:
* sliding window of width W keeps keys j with i - W < j <= i (W keys,
  diagonal included; W = 1 leaves only the diagonal);
* ALiBi is the additive bias -slope_h * (i - j) on the scaled score, indexed by
  query head h (slopes are an input);
* query head h reads K/V head h // (H / H_kv) (contiguous groups);
* a row with no visible key gets O = 0 and LSE = -inf;
* the softmax scale defaults to 1/sqrt(D); LSE is a natural logarithm;
* queries and keys share positions 0..S-1 (plus an optional common offset,
  which only moves the RoPE angles);
* the additive bias is a tensor broadcastable to [B, H, S, S] (query head h),
  added after the scale and before the mask, exactly like ALiBi;
* relu attention is P = max(s, 0) with no normalisation (a 1/n factor such as
  dividing by the sequence length folds into the scale and the bias, since
  max(a s, 0) = a max(s, 0) for a > 0).
"""
import numpy as np

from .rope import ROPE_NONE, rope_rotate

MASK_NONE = "none"
MASK_CAUSAL = "causal"
MASK_SLIDING_WINDOW = "sliding_window"
MASK_KINDS = (MASK_NONE, MASK_CAUSAL, MASK_SLIDING_WINDOW)
NORM_SOFTMAX = "softmax"
NORM_RELU = "relu"
NORM_KINDS = (NORM_SOFTMAX, NORM_RELU)

# Rows per chunk when a head's score matrix would not fit comfortably in memory.
_ROW_CHUNK = 2048


def block_visible(i, j, block_mask):
    """Block-sparse mask (Section 4.3 "Block-Sparse Attention"): block_mask is
    (block_size, active) with active[qb, kb] True when query block qb may see key
    block kb.  Returns the boolean matrix for query positions i, key positions j."""
    bs, active = block_mask
    active = np.asarray(active, dtype=bool)
    return active[np.asarray(i)[:, None] // bs, np.asarray(j)[None, :] // bs]


def visibility(i, j, mask, window=None, block_mask=None):
    """Boolean matrix: is key j visible to query i (i, j index arrays, broadcast).

    With a block mask, a key is visible when both the elementwise mask and its
    block allow it."""
    i = np.asarray(i)
    j = np.asarray(j)
    ii = i[:, None]
    jj = j[None, :]
    if mask == MASK_NONE:
        vis = np.ones((ii.shape[0], jj.shape[1]), dtype=bool)
    elif mask == MASK_CAUSAL:
        vis = jj <= ii
    elif mask == MASK_SLIDING_WINDOW:
        if window is None or window < 1:
            raise ValueError("sliding window needs window >= 1")
        vis = (jj <= ii) & (jj > ii - window)
    else:
        raise ValueError(f"unknown mask {mask!r}")
    if block_mask is not None:
        vis = vis & block_visible(i, j, block_mask)
    return vis


def kv_head(h, H, Hkv):
    """K/V head read by query head h: contiguous groups of H/H_kv query heads."""
    return h // (H // Hkv)


def alibi_bias(slope, rows, cols):
    """ALiBi bias -slope * (i - j) for query positions ``rows`` and key positions ``cols``."""
    return -slope * (np.asarray(rows)[:, None] - np.asarray(cols)[None, :]).astype(np.float64)


def _check(q, k, v):
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("q, k, v must be [B, heads, S, D]")
    B, H, S, D = q.shape
    if k.shape[0] != B or k.shape[2:] != (S, D) or v.shape != k.shape:
        raise ValueError("k and v must be [B, H_kv, S, D] matching q")
    Hkv = k.shape[1]
    if H % Hkv:
        raise ValueError("H must be a multiple of H_kv")
    return B, H, Hkv, S, D


def _rotated(q, k, rope, theta, pos_offset):
    S = q.shape[2]
    pos = np.arange(S, dtype=np.float64) + pos_offset
    return rope_rotate(q, pos, theta, rope), rope_rotate(k, pos, theta, rope)


def attention_scores(qr_bh, kr_bg, rows, *, mask, window, slope, scale, block_mask=None, bias_bh=None):
    """Step 2-3 for one (b, h): scaled scores of the given query rows with bias and mask.

    qr_bh [S, D], kr_bg [S, D] already rotated; bias_bh [S, S] or None.
    Returns [len(rows), S] fp64 with masked entries at -inf.
    """
    S = kr_bg.shape[0]
    rows = np.asarray(rows)
    cols = np.arange(S)
    s = scale * (qr_bh[rows] @ kr_bg.T)
    if slope is not None:
        s = s + alibi_bias(slope, rows, cols)
    if bias_bh is not None:
        s = s + bias_bh[rows]
    vis = visibility(rows, cols, mask, window, block_mask)
    return np.where(vis, s, -np.inf)


def _relu_rows(s):
    """Step 4 under relu attention: P = max(s, 0); masked entries (-inf) give 0."""
    return np.maximum(s, 0.0)


def _relu_grad(s, dP):
    """dS under relu attention: dP where the score is positive, else 0."""
    return np.where(s > 0.0, dP, 0.0)


def _bias_of(bias, B, H, S):
    """The bias tensor broadcast to [B, H, S, S] (a read-only view), or None."""
    if bias is None:
        return None
    bias = np.asarray(bias, dtype=np.float64)
    try:
        return np.broadcast_to(bias, (B, H, S, S))
    except ValueError:
        raise ValueError("bias must broadcast to [B, H, S, S]") from None


def _norm_of(norm):
    if norm not in NORM_KINDS:
        raise ValueError(f"unknown norm {norm!r}")
    return norm


def _softmax_rows(s):
    """Step 4: returns (P, m, l); rows with no visible key give P = 0, m = -inf, l = 0."""
    m = np.max(s, axis=1)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    e = np.exp(s - m_safe[:, None])          # exp(-inf) = 0 for masked entries
    l = np.sum(e, axis=1)
    P = np.where(finite[:, None], e / np.where(finite, l, 1.0)[:, None], 0.0)
    return P, m, np.where(finite, l, 0.0)


def _defaults(D, scale, alibi_slopes, H):
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    slopes = None
    if alibi_slopes is not None:
        slopes = np.asarray(alibi_slopes, dtype=np.float64)
        if slopes.shape != (H,):
            raise ValueError("alibi_slopes must have one slope per query head")
    return float(scale), slopes


def attention_probs(q, k, b, h, *, rope=ROPE_NONE, theta=10000.0, mask=MASK_CAUSAL,
                    window=None, alibi_slopes=None, scale=None, pos_offset=0, block_mask=None):
    """The full softmax matrix P [S, S] of one (b, h) (for invariant checks)."""
    B, H, Hkv, S, D = _check(q, k, k)
    scale, slopes = _defaults(D, scale, alibi_slopes, H)
    qr, kr = _rotated(q, k, rope, theta, pos_offset)
    g = kv_head(h, H, Hkv)
    s = attention_scores(qr[b, h], kr[b, g], np.arange(S), mask=mask, window=window,
                         slope=None if slopes is None else slopes[h], scale=scale, block_mask=block_mask)
    return _softmax_rows(s)[0]


def attention_forward(q, k, v, *, rope=ROPE_NONE, theta=10000.0, mask=MASK_CAUSAL,
                      window=None, alibi_slopes=None, scale=None, pos_offset=0, block_mask=None,
                      bias=None, norm=NORM_SOFTMAX):
    """O [B, H, S, D] and LSE [B, H, S] (natural log), both fp64; LSE is None
    under relu attention."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, Hkv, S, D = _check(q, k, v)
    scale, slopes = _defaults(D, scale, alibi_slopes, H)
    bias = _bias_of(bias, B, H, S)
    norm = _norm_of(norm)
    qr, kr = _rotated(q, k, rope, theta, pos_offset)
    O = np.zeros((B, H, S, D))
    LSE = np.empty((B, H, S))
    for b in range(B):
        for h in range(H):
            g = kv_head(h, H, Hkv)
            slope = None if slopes is None else slopes[h]
            for r0 in range(0, S, _ROW_CHUNK):
                rows = np.arange(r0, min(S, r0 + _ROW_CHUNK))
                s = attention_scores(qr[b, h], kr[b, g], rows, mask=mask, window=window,
                                     slope=slope, scale=scale, block_mask=block_mask,
                                     bias_bh=None if bias is None else bias[b, h])
                if norm == NORM_RELU:
                    O[b, h, rows] = _relu_rows(s) @ v[b, g]
                    continue
                P, m, l = _softmax_rows(s)
                O[b, h, rows] = P @ v[b, g]
                with np.errstate(divide="ignore"):
                    LSE[b, h, rows] = m + np.log(l)
    return O, (None if norm == NORM_RELU else LSE)


def attention_forward_rows(q_bh, k_bg, v_bg, rows, *, h=0, H=1, rope=ROPE_NONE,
                           theta=10000.0, mask=MASK_CAUSAL, window=None,
                           alibi_slopes=None, scale=None, pos_offset=0, block_mask=None,
                           bias_bh=None, norm=NORM_SOFTMAX):
    """O and LSE of selected query rows of ONE head, for sampled checks at full size.

    q_bh [S, D] is query head h; k_bg, v_bg [S, D] its K/V head.  Only the
    requested rows' scores are formed, so the cost is len(rows) * S * D.
    ``alibi_slopes`` is the full per-query-head slope vector (length H).
    """
    q_bh = np.asarray(q_bh, dtype=np.float64)
    k_bg = np.asarray(k_bg, dtype=np.float64)
    v_bg = np.asarray(v_bg, dtype=np.float64)
    S, D = k_bg.shape
    scale, slopes = _defaults(D, scale, alibi_slopes, H)
    pos = np.arange(S, dtype=np.float64) + pos_offset
    rows = np.asarray(rows)
    qr = rope_rotate(q_bh[rows], pos[rows], theta, rope)
    kr = rope_rotate(k_bg, pos, theta, rope)
    # Scores of the selected rows only (step 2-3 restricted to those rows).
    s = scale * (qr @ kr.T)
    cols = np.arange(S)
    if slopes is not None:
        s = s + alibi_bias(slopes[h], rows, cols)
    if bias_bh is not None:
        s = s + np.asarray(bias_bh, dtype=np.float64)[rows]
    s = np.where(visibility(rows, cols, mask, window, block_mask), s, -np.inf)
    if _norm_of(norm) == NORM_RELU:
        return _relu_rows(s) @ v_bg, None
    P, m, l = _softmax_rows(s)
    with np.errstate(divide="ignore"):
        return P @ v_bg, m + np.log(l)


def _row_delta(P, dP, dO_rows, o_rows):
    """delta_i of the softmax backward: sum_j P_ij dP_ij, or rowsum(dO_i * o_i)
    of a given forward output (equal for the exact output)."""
    if o_rows is None:
        return np.sum(P * dP, axis=1)
    return np.sum(dO_rows * o_rows, axis=1)


def attention_backward(q, k, v, do, *, rope=ROPE_NONE, theta=10000.0, mask=MASK_CAUSAL,
                       window=None, alibi_slopes=None, scale=None, pos_offset=0,
                       return_intermediates=False, block_mask=None, bias=None, norm=NORM_SOFTMAX,
                       relu_gate="exact", o=None):
    """dQ [B,H,S,D], dK and dV [B,H_kv,S,D] in fp64.

    With ``return_intermediates`` also returns a dict with per-(b,h) lists of
    P, dS and delta (only sensible at small sizes; delta is absent under relu
    attention).

    ``relu_gate`` says in which precision the relu derivative's decision
    s > 0 is taken: "exact" (fp64, the definition) or "fp16" (the score formed
    from the rotated Q' and K' rounded to fp16, the operand precision of an
    fp16 matrix unit).  The gate is a discontinuous function of the score, so a
    score within rounding of 0 flips it; comparing against a kernel that gates
    on fp16 operands takes the decision in that precision on both sides.
    Everything else stays fp64.

    ``o`` [B,H,S,D] is the forward output the backward is given.  The softmax
    backward's row term delta_i = sum_j P_ij dP_ij equals rowsum(dO_i * O_i)
    for the exact O, and the three-pass backward (Section 4.4) forms it in its
    preprocessing pass from the O it receives; with ``o`` given, delta is
    rowsum(dO_i * o_i) of that array (in fp64), so a caller's rounded O enters
    exactly as it does there.  None (the default) uses the definitional sum.
    Unused under relu attention (no delta).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    B, H, Hkv, S, D = _check(q, k, v)
    if do.shape != q.shape:
        raise ValueError("dO must have the shape of Q")
    if o is not None:
        o = np.asarray(o, dtype=np.float64)
        if o.shape != q.shape:
            raise ValueError("O must have the shape of Q")
    scale, slopes = _defaults(D, scale, alibi_slopes, H)
    bias = _bias_of(bias, B, H, S)
    norm = _norm_of(norm)
    if relu_gate not in ("exact", "fp16"):
        raise ValueError(f"unknown relu_gate {relu_gate!r}")
    qr, kr = _rotated(q, k, rope, theta, pos_offset)
    if relu_gate == "fp16":
        qg = qr.astype(np.float16).astype(np.float64)
        kg = kr.astype(np.float16).astype(np.float64)
    dqr = np.zeros_like(qr)
    dkr = np.zeros_like(kr)
    dv = np.zeros_like(v)
    inter = {"P": {}, "dS": {}, "delta": {}}
    for b in range(B):
        for h in range(H):
            g = kv_head(h, H, Hkv)
            slope = None if slopes is None else slopes[h]
            for r0 in range(0, S, _ROW_CHUNK):
                rows = np.arange(r0, min(S, r0 + _ROW_CHUNK))
                s = attention_scores(qr[b, h], kr[b, g], rows, mask=mask, window=window,
                                     slope=slope, scale=scale, block_mask=block_mask,
                                     bias_bh=None if bias is None else bias[b, h])
                P = _relu_rows(s) if norm == NORM_RELU else _softmax_rows(s)[0]
                dO_rows = do[b, h, rows]
                dv[b, g] += P.T @ dO_rows
                dP = dO_rows @ v[b, g].T
                if norm == NORM_RELU:
                    delta = None
                    sg = s
                    if relu_gate == "fp16":
                        sg = attention_scores(qg[b, h], kg[b, g], rows, mask=mask, window=window, slope=slope,
                                              scale=scale, block_mask=block_mask,
                                              bias_bh=None if bias is None else bias[b, h])
                    dS = _relu_grad(sg, dP)
                else:
                    delta = _row_delta(P, dP, dO_rows, None if o is None else o[b, h, rows])
                    dS = P * (dP - delta[:, None])
                dqr[b, h, rows] = scale * (dS @ kr[b, g])
                dkr[b, g] += scale * (dS.T @ qr[b, h, rows])
                if return_intermediates and S <= _ROW_CHUNK:
                    inter["P"][(b, h)] = P
                    inter["dS"][(b, h)] = dS
                    inter["delta"][(b, h)] = delta
    pos = np.arange(S, dtype=np.float64) + pos_offset
    dq = rope_rotate(dqr, pos, theta, rope, inverse=True)
    dk = rope_rotate(dkr, pos, theta, rope, inverse=True)
    if return_intermediates:
        return dq, dk, dv, inter
    return dq, dk, dv
