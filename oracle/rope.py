"""RoPE (rotary position embedding) in fp64 -- oracle, test infrastructure only.

Section 2 ("Rotary Position Embeddings"): each pair of dimensions of a query or
key vector is rotated by an angle proportional to the token's position, which
makes the rotated dot product depend only on the relative position.  Section
4.1 ("Fused RoPE") fixes the pairing as the NeoX convention, where a dimension
is paired with the one half a head-dimension away ("the rotated half").  The
small parity workload instead asks for interleaved pairs (2i, 2i+1), so both
pairings are provided.

Readings of points the paper leaves open:
* frequencies: omega_i = theta^(-2i/D) for pair index i in [0, D/2), the
  RoFormer definition the paper cites;
* sign: the second element of each pair gets +sin, i.e.
  x'_a = x_a cos(a) - x_b sin(a),  x'_b = x_a sin(a) + x_b cos(a);
* positions are 0..S-1 for both queries and keys unless an offset is given.
"""
import numpy as np

ROPE_NONE = "none"
ROPE_NEOX = "neox"
ROPE_INTERLEAVED = "interleaved"
ROPE_KINDS = (ROPE_NONE, ROPE_NEOX, ROPE_INTERLEAVED)


def rope_frequencies(D, theta):
    """Angular frequency of each of the D/2 pairs: omega_i = theta^(-2i/D), fp64."""
    if D % 2:
        raise ValueError("RoPE needs an even head dimension")
    i = np.arange(D // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * i / D)


def rope_pair_indices(D, kind):
    """(a, b): the two dimension indices of every pair i, in pair order.

    NeoX (Section 4.1): pair i is (i, i + D/2).  Interleaved: (2i, 2i + 1).
    """
    half = D // 2
    i = np.arange(half)
    if kind == ROPE_NEOX:
        return i, i + half
    if kind == ROPE_INTERLEAVED:
        return 2 * i, 2 * i + 1
    raise ValueError(f"no pairing for rope kind {kind!r}")


def rope_rotate(x, positions, theta, kind, inverse=False):
    """Rotate every pair of the last axis of ``x`` by position * omega_i.

    x: array [..., S, D] (any float dtype; computed in fp64).
    positions: integer or float array [S].
    inverse: rotate by the negative angle, i.e. apply R^T = R^-1 (used for the
    gradient of the rotation, which is orthogonal).
    Returns a new fp64 array; kind == "none" returns an fp64 copy.
    """
    x = np.asarray(x, dtype=np.float64)
    if kind == ROPE_NONE:
        return x.copy()
    S, D = x.shape[-2], x.shape[-1]
    positions = np.asarray(positions, dtype=np.float64)
    if positions.shape != (S,):
        raise ValueError("positions must have one entry per sequence position")
    angle = positions[:, None] * rope_frequencies(D, theta)[None, :]   # [S, D/2]
    if inverse:
        angle = -angle
    c = np.cos(angle)
    s = np.sin(angle)
    a, b = rope_pair_indices(D, kind)
    xa = x[..., a]
    xb = x[..., b]
    out = np.empty_like(x)
    out[..., a] = xa * c - xb * s
    out[..., b] = xa * s + xb * c
    return out
