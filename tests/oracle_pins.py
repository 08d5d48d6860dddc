"""Checks that pin the fp64 oracle to things other than itself.

Each ``check_*`` raises AssertionError on failure.  They are run as tests in
``test_oracle_pins.py`` and, with a mistake planted in the oracle, in
``test_oracle_mutations.py`` (which asserts that some check then fails).

Sources of truth used here, none of them the oracle:
* closed forms (D = 2 rotations, frequencies of a tiny head, the first rows of
  a causal softmax, a width-1 window);
* invariants of the definitions (rotation norms, relative-position dot
  products, softmax rows summing to one, rows of dS summing to zero);
* an independent brute force (tests/bruteforce.py: explicit Givens matrices and
  scalar loops) and its finite-difference gradients;
* library routines: torch's fp64 scaled_dot_product_attention on the CPU, and
  torch autograd through a separately written torch forward that applies RoPE
  as complex multiplication.
"""
import math

import numpy as np
import torch

import oracle
import bruteforce

TOL = 1e-12


def _rng(seed):
    return np.random.default_rng(seed)


def _tiny(seed, B=1, H=2, Hkv=1, S=6, D=4):
    r = _rng(seed)
    q = r.standard_normal((B, H, S, D))
    k = r.standard_normal((B, Hkv, S, D))
    v = r.standard_normal((B, Hkv, S, D))
    do = r.standard_normal((B, H, S, D))
    return q, k, v, do


# ----------------------------------------------------------------------------- RoPE

def check_frequencies():
    w = oracle.rope_frequencies(8, 10000.0)
    assert np.allclose(w, [1.0, 0.1, 0.01, 0.001], rtol=1e-14, atol=0)
    w = oracle.rope_frequencies(128, 500000.0)
    assert w[0] == 1.0
    assert abs(w[1] - 500000.0 ** (-1.0 / 64.0)) < 1e-16


def check_rope_d2_closed_form(kind):
    p = 3.0   # D = 2 has one pair with omega_0 = 1, so the angle is p radians
    x = np.array([[1.0, 0.0], [0.0, 1.0]])   # two "positions" sharing p
    out = oracle.rope_rotate(x, np.array([p, p]), 10000.0, kind)
    assert np.allclose(out[0], [math.cos(p), math.sin(p)], atol=1e-15)
    assert np.allclose(out[1], [-math.sin(p), math.cos(p)], atol=1e-15)


def check_rope_pairing(kind):
    D, p = 8, 5.0
    partner = {"neox": lambda a: (a + D // 2) % D, "interleaved": lambda a: a ^ 1}[kind]
    for a in range(D):
        x = np.zeros((1, D))
        x[0, a] = 1.0
        out = oracle.rope_rotate(x, np.array([p]), 7.0, kind)[0]
        nz = set(np.flatnonzero(np.abs(out) > 1e-14).tolist())
        assert nz == {a, partner(a)}, (kind, a, nz)


def check_rope_norm(kind, seed=1):
    x = _rng(seed).standard_normal((2, 3, 50, 16))
    pos = np.arange(50) * 37.0
    out = oracle.rope_rotate(x, pos, 10000.0, kind)
    a, b = {"neox": (np.arange(8), np.arange(8) + 8),
            "interleaved": (np.arange(0, 16, 2), np.arange(1, 16, 2))}[kind]
    assert np.allclose(out[..., a] ** 2 + out[..., b] ** 2, x[..., a] ** 2 + x[..., b] ** 2, atol=1e-12)
    assert np.allclose(np.linalg.norm(out, axis=-1), np.linalg.norm(x, axis=-1), atol=1e-12)


def check_rope_relative(kind, seed=2):
    r = _rng(seed)
    q = r.standard_normal(16)
    k = r.standard_normal(16)
    for (m, n, t) in [(5, 2, 11), (0, 9, 100), (300, 1, 7)]:
        def rot(x, p):
            return oracle.rope_rotate(x[None], np.array([float(p)]), 10000.0, kind)[0]
        base = rot(q, m) @ rot(k, n)
        shifted = rot(q, m + t) @ rot(k, n + t)
        assert abs(base - shifted) < 1e-12
    # and it is not position-blind: a different offset changes the product
    assert abs(rot(q, 5) @ rot(k, 2) - rot(q, 5) @ rot(k, 3)) > 1e-6


def check_rope_inverse(kind, seed=3):
    x = _rng(seed).standard_normal((4, 32))
    pos = np.arange(4) * 1000.0
    y = oracle.rope_rotate(x, pos, 500000.0, kind)
    assert np.allclose(oracle.rope_rotate(y, pos, 500000.0, kind, inverse=True), x, atol=1e-12)
    assert np.allclose(oracle.rope_rotate(x, np.zeros(4), 500000.0, kind), x, atol=0)


def check_rope_vs_givens(kind, seed=4):
    D, S = 8, 5
    x = _rng(seed).standard_normal((S, D))
    pos = np.arange(S) + 3.0
    out = oracle.rope_rotate(x, pos, 10000.0, kind)
    for s in range(S):
        R = bruteforce.givens_matrix(D, pos[s], 10000.0, kind)
        assert np.allclose(out[s], bruteforce.matvec(R, list(x[s])), atol=1e-13)


# ----------------------------------------------------------------------------- forward

VARIANTS = [
    # (rope, mask, window, alibi)
    ("none", "none", None, False),
    ("none", "causal", None, False),
    ("neox", "causal", None, False),
    ("interleaved", "causal", None, False),
    ("neox", "none", None, False),
    ("neox", "sliding_window", 3, False),
    ("interleaved", "sliding_window", 1, False),
    ("none", "causal", None, True),
    ("neox", "causal", None, True),
    ("neox", "sliding_window", 2, True),
]


def _kw(rope, mask, window, alibi, H):
    slopes = [0.3 * (h + 1) for h in range(H)] if alibi else None
    return dict(rope=rope, theta=10000.0, mask=mask, window=window, alibi_slopes=slopes, scale=0.41)


def check_forward_vs_bruteforce(variant, seed=5):
    rope, mask, window, alibi = variant
    q, k, v, _ = _tiny(seed, B=2, H=4, Hkv=2, S=7, D=4)
    kw = _kw(rope, mask, window, alibi, 4)
    O, L = oracle.attention_forward(q, k, v, **kw)
    Ob, Lb = bruteforce.forward(q.tolist(), k.tolist(), v.tolist(), **kw)
    assert np.allclose(O, np.array(Ob), atol=TOL, rtol=0)
    assert np.allclose(L, np.array(Lb), atol=TOL, rtol=0)


def check_softmax_rows(variant, seed=6):
    rope, mask, window, alibi = variant
    q, k, v, _ = _tiny(seed, H=2, Hkv=2, S=9, D=8)
    kw = _kw(rope, mask, window, alibi, 2)
    for h in range(2):
        P = oracle.attention_probs(q, k, 0, h, **kw)
        assert np.allclose(P.sum(axis=1), 1.0, atol=1e-14)
        assert (P >= 0).all()
        i = np.arange(9)[:, None]
        j = np.arange(9)[None, :]
        if mask == "causal":
            assert (P[j > i] == 0).all()
        if mask == "sliding_window":
            assert (P[(j > i) | (j <= i - window)] == 0).all()


def check_causal_first_rows(kind, seed=7):
    # Row 0 sees only key 0 and RoPE is the identity at position 0, so
    # O_0 = v_0 and LSE_0 = scale * q_0 . k_0.
    q, k, v, _ = _tiny(seed, H=1, Hkv=1, S=5, D=2)
    scale = 0.8
    O, L = oracle.attention_forward(q, k, v, rope=kind, mask="causal", scale=scale)
    assert np.allclose(O[0, 0, 0], v[0, 0, 0], atol=1e-15)
    assert abs(L[0, 0, 0] - scale * q[0, 0, 0] @ k[0, 0, 0]) < 1e-14
    # Row 1 (D = 2, omega = 1): q_1 rotated by 1 rad against k_0 (unrotated) and
    # k_1 (rotated by the same 1 rad, so that product is rotation-free).
    if kind != "none":
        c, s = math.cos(1.0), math.sin(1.0)
        q1 = q[0, 0, 1]
        q1r = np.array([q1[0] * c - q1[1] * s, q1[0] * s + q1[1] * c])
        s10 = scale * q1r @ k[0, 0, 0]
        s11 = scale * q1 @ k[0, 0, 1]
        e0, e1 = math.exp(s10), math.exp(s11)
        assert np.allclose(O[0, 0, 1], (e0 * v[0, 0, 0] + e1 * v[0, 0, 1]) / (e0 + e1), atol=1e-14)
        assert abs(L[0, 0, 1] - math.log(e0 + e1)) < 1e-14


def check_window_one(kind, seed=8):
    # Width-1 window: each row sees only itself, so O = V and, because both
    # sides rotate by the same angle, LSE_i = scale * q_i . k_i.
    q, k, v, _ = _tiny(seed, H=2, Hkv=2, S=10, D=8)
    O, L = oracle.attention_forward(q, k, v, rope=kind, mask="sliding_window", window=1, scale=0.5)
    assert np.allclose(O, v, atol=1e-15)
    assert np.allclose(L, 0.5 * np.einsum("bhsd,bhsd->bhs", q, k), atol=1e-13)


def check_window_reductions(seed=9):
    q, k, v, _ = _tiny(seed, H=2, Hkv=1, S=12, D=8)
    causal = oracle.attention_forward(q, k, v, rope="neox", mask="causal")
    for W in (12, 13, 100):
        sw = oracle.attention_forward(q, k, v, rope="neox", mask="sliding_window", window=W)
        assert np.allclose(sw[0], causal[0], atol=1e-14) and np.allclose(sw[1], causal[1], atol=1e-14)
    # a window of 11 differs from causal only in rows that can see 12 keys
    sw = oracle.attention_forward(q, k, v, rope="neox", mask="sliding_window", window=11)
    assert np.allclose(sw[0][:, :, :11], causal[0][:, :, :11], atol=1e-14)
    assert not np.allclose(sw[0][:, :, 11], causal[0][:, :, 11], atol=1e-6)


def check_alibi_special_cases(seed=10):
    q, k, v, _ = _tiny(seed, H=3, Hkv=3, S=8, D=4)
    plain = oracle.attention_forward(q, k, v, rope="neox", mask="causal")
    zero = oracle.attention_forward(q, k, v, rope="neox", mask="causal", alibi_slopes=[0.0] * 3)
    assert np.allclose(plain[0], zero[0], atol=1e-15) and np.allclose(plain[1], zero[1], atol=1e-15)
    # A huge slope makes every earlier key vanish: O -> V and LSE -> the diagonal score.
    big = oracle.attention_forward(q, k, v, rope="neox", mask="causal", alibi_slopes=[1e3] * 3)
    assert np.allclose(big[0], v, atol=1e-12)
    assert np.allclose(big[1], 0.5 * np.einsum("bhsd,bhsd->bhs", q, k), atol=1e-12)
    # Row 1 with two visible keys: the earlier key is penalised by exactly one slope.
    s = 0.7
    one = oracle.attention_forward(q, k, v, mask="causal", alibi_slopes=[s] * 3, scale=0.5)
    s10 = 0.5 * q[0, 0, 1] @ k[0, 0, 0] - s
    s11 = 0.5 * q[0, 0, 1] @ k[0, 0, 1]
    assert abs(one[1][0, 0, 1] - math.log(math.exp(s10) + math.exp(s11))) < 1e-13


def check_vs_torch_sdpa(mask, seed=11):
    q, k, v, _ = _tiny(seed, B=2, H=3, Hkv=3, S=33, D=16)
    O, _ = oracle.attention_forward(q, k, v, rope="none", mask=mask, scale=0.3)
    t = [torch.from_numpy(x) for x in (q, k, v)]
    ref = torch.nn.functional.scaled_dot_product_attention(*t, is_causal=(mask == "causal"), scale=0.3)
    assert np.allclose(O, ref.numpy(), atol=1e-12)


def check_position_shift(kind, mask, seed=12):
    q, k, v, _ = _tiny(seed, H=2, Hkv=1, S=10, D=8)
    kw = dict(rope=kind, mask=mask, window=4 if mask == "sliding_window" else None, alibi_slopes=[0.2, 0.1])
    a = oracle.attention_forward(q, k, v, **kw)
    b = oracle.attention_forward(q, k, v, pos_offset=1234, **kw)
    assert np.allclose(a[0], b[0], atol=1e-10) and np.allclose(a[1], b[1], atol=1e-10)


def check_gqa_repeat_kv(seed=13):
    q, k, v, do = _tiny(seed, B=2, H=6, Hkv=2, S=7, D=8)
    kw = dict(rope="neox", mask="causal", alibi_slopes=[0.1 * h for h in range(6)])
    O, L = oracle.attention_forward(q, k, v, **kw)
    kr = np.repeat(k, 3, axis=1)   # HF repeat_kv: query head h reads K/V head h // 3
    vr = np.repeat(v, 3, axis=1)
    O2, L2 = oracle.attention_forward(q, kr, vr, **kw)
    assert np.allclose(O, O2, atol=1e-15) and np.allclose(L, L2, atol=1e-15)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, **kw)
    dq2, dk2, dv2 = oracle.attention_backward(q, kr, vr, do, **kw)
    assert np.allclose(dq, dq2, atol=1e-13)
    assert np.allclose(dk, dk2.reshape(2, 2, 3, 7, 8).sum(axis=2), atol=1e-13)
    assert np.allclose(dv, dv2.reshape(2, 2, 3, 7, 8).sum(axis=2), atol=1e-13)


def check_rows_match_full(seed=14):
    q, k, v, _ = _tiny(seed, B=1, H=4, Hkv=2, S=40, D=8)
    slopes = [0.05, 0.1, 0.2, 0.4]
    for rope, mask, W in [("neox", "causal", None), ("interleaved", "sliding_window", 5), ("none", "none", None)]:
        O, L = oracle.attention_forward(q, k, v, rope=rope, mask=mask, window=W, alibi_slopes=slopes)
        rows = np.array([0, 3, 17, 39])
        for h in range(4):
            o, l = oracle.attention_forward_rows(q[0, h], k[0, h // 2], v[0, h // 2], rows, h=h, H=4,
                                                 rope=rope, mask=mask, window=W, alibi_slopes=slopes)
            assert np.allclose(o, O[0, h, rows], atol=1e-14) and np.allclose(l, L[0, h, rows], atol=1e-14)


# ----------------------------------------------------------------------------- backward

def check_backward_fd(variant, seed=15):
    rope, mask, window, alibi = variant
    q, k, v, do = _tiny(seed, B=1, H=2, Hkv=1, S=5, D=4)
    kw = _kw(rope, mask, window, alibi, 2)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, **kw)
    ql, kl, vl, dol = q.tolist(), k.tolist(), v.tolist(), do.tolist()

    def f():
        return bruteforce.loss(ql, kl, vl, dol, **kw)

    assert np.allclose(dq, np.array(bruteforce.finite_difference_grad(ql, f)), atol=1e-7)
    assert np.allclose(dk, np.array(bruteforce.finite_difference_grad(kl, f)), atol=1e-7)
    assert np.allclose(dv, np.array(bruteforce.finite_difference_grad(vl, f)), atol=1e-7)


def _torch_forward(q, k, v, rope, mask, window, slopes, scale, theta):
    """A separately written torch fp64 forward: RoPE as complex multiplication."""
    B, H, S, D = q.shape
    Hkv = k.shape[1]
    pos = torch.arange(S, dtype=torch.float64)
    inv = theta ** (-torch.arange(0, D, 2, dtype=torch.float64) / D)
    phase = torch.polar(torch.ones(S, D // 2, dtype=torch.float64), pos[:, None] * inv[None, :])

    def rot(x):
        if rope == "none":
            return x
        if rope == "interleaved":
            z = torch.view_as_complex(x.reshape(*x.shape[:-1], D // 2, 2))
            return torch.view_as_real(z * phase).reshape(x.shape)
        z = torch.complex(x[..., : D // 2], x[..., D // 2:])
        z = z * phase
        return torch.cat([z.real, z.imag], dim=-1)

    qr, kr = rot(q), rot(k)
    kr = kr.repeat_interleave(H // Hkv, dim=1)
    vv = v.repeat_interleave(H // Hkv, dim=1)
    s = scale * qr @ kr.transpose(-1, -2)
    i = torch.arange(S)[:, None]
    j = torch.arange(S)[None, :]
    if slopes is not None:
        s = s + torch.tensor(slopes, dtype=torch.float64)[None, :, None, None] * (j - i).to(torch.float64)
    keep = torch.ones(S, S, dtype=torch.bool)
    if mask in ("causal", "sliding_window"):
        keep &= j <= i
    if mask == "sliding_window":
        keep &= (i - j) < window
    s = s.masked_fill(~keep, float("-inf"))
    return torch.softmax(s, dim=-1) @ vv


def check_backward_vs_torch_autograd(variant, seed=16):
    rope, mask, window, alibi = variant
    q, k, v, do = _tiny(seed, B=2, H=4, Hkv=2, S=11, D=8)
    kw = _kw(rope, mask, window, alibi, 4)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, **kw)
    O, _ = oracle.attention_forward(q, k, v, **kw)
    t = [torch.tensor(x, requires_grad=True) for x in (q, k, v)]
    out = _torch_forward(*t, rope, mask, window, kw["alibi_slopes"], kw["scale"], kw["theta"])
    assert np.allclose(out.detach().numpy(), O, atol=1e-12)
    out.backward(torch.from_numpy(do))
    assert np.allclose(t[0].grad.numpy(), dq, atol=1e-12)
    assert np.allclose(t[1].grad.numpy(), dk, atol=1e-12)
    assert np.allclose(t[2].grad.numpy(), dv, atol=1e-12)


def check_backward_identities(seed=17):
    q, k, v, do = _tiny(seed, B=1, H=2, Hkv=2, S=9, D=8)
    kw = dict(rope="neox", mask="causal", alibi_slopes=[0.3, 0.6])
    dq, dk, dv, inter = oracle.attention_backward(q, k, v, do, return_intermediates=True, **kw)
    O, _ = oracle.attention_forward(q, k, v, **kw)
    for h in range(2):
        dS = inter["dS"][(0, h)]
        assert np.allclose(dS.sum(axis=1), 0.0, atol=1e-13)          # softmax Jacobian rows
        assert np.allclose(inter["delta"][(0, h)], (do[0, h] * O[0, h]).sum(axis=1), atol=1e-13)
    # Causal row 0 only sees key 0 with weight 1: its query gradient is zero.
    assert np.allclose(dq[:, :, 0], 0.0, atol=1e-14)
    # The last key is seen only by the last query: dV_{S-1} = sum over heads of P * dO.
    P_last = [inter["P"][(0, h)][-1, -1] for h in range(2)]
    assert np.allclose(dv[0, :, -1], np.array([P_last[h] * do[0, h, -1] for h in range(2)]), atol=1e-13)


# ----------------------------------------------------------------------------- decode

def _decode_case(seed, B=2, H=4, Hkv=2, S=7, D=4):
    r = _rng(seed)
    return (r.standard_normal((B, H, D)), r.standard_normal((B, Hkv, S, D)), r.standard_normal((B, Hkv, S, D)))


def check_decode_vs_bruteforce(variant, seed=20):
    rope, mask, window, alibi = variant
    q, kc, vc = _decode_case(seed)
    kw = _kw(rope, mask, window, alibi, 4)
    for lens in (None, [7, 3]):
        O, L = oracle.decode_forward(q, kc, vc, lens, **kw)
        Ob, Lb = bruteforce.decode(q.tolist(), kc.tolist(), vc.tolist(), lens, **kw)
        assert np.allclose(O, np.array(Ob), atol=TOL, rtol=0)
        assert np.allclose(L, np.array(Lb), atol=TOL, rtol=0)


def check_decode_is_last_prefill_row(variant, seed=21):
    # A cache written with keys rotated at their own positions, queried by the
    # last token, is the last row of the prefill attention over those tokens.
    rope, mask, window, alibi = variant
    q, k, v, _ = _tiny(seed, B=2, H=4, Hkv=2, S=9, D=8)
    kw = _kw(rope, mask, window, alibi, 4)
    k_cache = oracle.rope_rotate(k, np.arange(9), 10000.0, rope)
    for n in (9, 5, 1):
        O, L = oracle.attention_forward(q[:, :, :n], k[:, :, :n], v[:, :, :n], **kw)
        Od, Ld = oracle.decode_forward(q[:, :, n - 1], k_cache, v, [n, n], **kw)
        assert np.allclose(Od, O[:, :, n - 1], atol=1e-13, rtol=0)
        assert np.allclose(Ld, L[:, :, n - 1], atol=1e-13, rtol=0)


def check_decode_closed_forms(kind, seed=22):
    q, kc, vc = _decode_case(seed, B=1, H=2, Hkv=2, S=6, D=8)
    # one cached token: the query is at position 0 (no rotation), O = v_0
    O, L = oracle.decode_forward(q, kc, vc, [1], rope=kind, scale=0.7)
    assert np.allclose(O[0], vc[0, :, 0], atol=1e-15)
    assert np.allclose(L[0], 0.7 * np.einsum("hd,hd->h", q[0], kc[0, :, 0]), atol=1e-14)
    # a width-1 window sees only the newest key
    O, _ = oracle.decode_forward(q, kc, vc, [5], rope=kind, mask="sliding_window", window=1)
    assert np.allclose(O[0], vc[0, :, 4], atol=1e-15)


def check_decode_ignores_stale_entries(seed=23):
    q, kc, vc = _decode_case(seed)
    base = oracle.decode_forward(q, kc, vc, [4, 6], rope="neox")
    kc2, vc2 = kc.copy(), vc.copy()
    kc2[0, :, 4:] = 1e3
    vc2[0, :, 4:] = -7.0
    kc2[1, :, 6:] = 5.0
    other = oracle.decode_forward(q, kc2, vc2, [4, 6], rope="neox")
    assert np.array_equal(base[0], other[0]) and np.array_equal(base[1], other[1])


# ----------------------------------------------------------------------------- block-sparse mask

def _random_blocks(seed, nb, density=0.45, empty_row=1):
    active = _rng(seed).random((nb, nb)) < density
    active[empty_row] = False              # a query block that sees nothing: O = 0, LSE = -inf
    return active


def check_block_mask_vs_bruteforce(variant, seed=30):
    rope, mask, window, alibi = variant
    q, k, v, _ = _tiny(seed, B=1, H=4, Hkv=2, S=9, D=4)
    kw = _kw(rope, mask, window, alibi, 4)
    bm = (2, _random_blocks(seed, 5))      # 2x2 blocks, the last one ragged
    O, L = oracle.attention_forward(q, k, v, block_mask=bm, **kw)
    Ob, Lb = bruteforce.forward(q.tolist(), k.tolist(), v.tolist(), block_mask=(bm[0], bm[1].tolist()), **kw)
    Ob, Lb = np.array(Ob), np.array(Lb)
    assert np.array_equal(np.isneginf(L), np.isneginf(Lb))
    fin = np.isfinite(Lb)
    assert np.allclose(L[fin], Lb[fin], atol=TOL, rtol=0)
    assert np.allclose(O, Ob, atol=TOL, rtol=0)
    assert np.isneginf(L[:, :, 2:4]).all() and (O[:, :, 2:4] == 0).all()   # block row 1 is empty


def check_block_mask_reductions(seed=31):
    q, k, v, do = _tiny(seed, B=1, H=2, Hkv=1, S=10, D=8)
    full = (4, np.ones((3, 3), dtype=bool))
    for mask in ("none", "causal"):
        a = oracle.attention_forward(q, k, v, rope="neox", mask=mask)
        b = oracle.attention_forward(q, k, v, rope="neox", mask=mask, block_mask=full)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
        ga = oracle.attention_backward(q, k, v, do, rope="neox", mask=mask)
        gb = oracle.attention_backward(q, k, v, do, rope="neox", mask=mask, block_mask=full)
        assert all(np.array_equal(x, y) for x, y in zip(ga, gb))
    # block-lower-triangular blocks under a causal mask are exactly causal
    tril = (4, np.tril(np.ones((3, 3), dtype=bool)))
    a = oracle.attention_forward(q, k, v, rope="interleaved", mask="causal")
    b = oracle.attention_forward(q, k, v, rope="interleaved", mask="causal", block_mask=tril)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def check_block_mask_backward_fd(seed=32):
    q, k, v, do = _tiny(seed, B=1, H=2, Hkv=1, S=6, D=4)
    active = _random_blocks(seed, 3, density=0.6, empty_row=2)
    active[0, 0] = active[1, 1] = True
    kw = dict(rope="neox", theta=10000.0, mask="none", window=None, alibi_slopes=None, scale=0.6)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, block_mask=(2, active), **kw)
    ql, kl, vl, dol = q.tolist(), k.tolist(), v.tolist(), do.tolist()

    def f():
        return bruteforce.loss(ql, kl, vl, dol, block_mask=(2, active.tolist()), **kw)

    assert np.allclose(dq, np.array(bruteforce.finite_difference_grad(ql, f)), atol=1e-7)
    assert np.allclose(dk, np.array(bruteforce.finite_difference_grad(kl, f)), atol=1e-7)
    assert np.allclose(dv, np.array(bruteforce.finite_difference_grad(vl, f)), atol=1e-7)


# ----------------------------------------------------------------------------- additive bias, relu attention

def _bias(seed, B, H, S, scale=1.5):
    return scale * _rng(seed + 1000).standard_normal((B, H, S, S))


def check_bias_relu_vs_bruteforce(variant, norm, seed=40):
    """The dense bias tensor (and relu attention) against the pure-Python loops."""
    rope, mask, window, alibi = variant
    q, k, v, _ = _tiny(seed, B=2, H=4, Hkv=2, S=7, D=4)
    kw = _kw(rope, mask, window, alibi, 4)
    bias = _bias(seed, 2, 4, 7)
    O, L = oracle.attention_forward(q, k, v, bias=bias, norm=norm, **kw)
    Ob, Lb = bruteforce.forward(q.tolist(), k.tolist(), v.tolist(), bias=bias.tolist(), norm=norm, **kw)
    assert np.allclose(O, np.array(Ob), atol=TOL, rtol=0)
    if norm == "relu":
        assert L is None and Lb is None
    else:
        assert np.allclose(L, np.array(Lb), atol=TOL, rtol=0)


def check_bias_reductions(seed=41):
    """Special cases that reduce the bias to other parts of the definition:
    the ALiBi matrix as a bias tensor is ALiBi; -inf above the diagonal is the
    causal mask; a bias constant along each row leaves O unchanged and shifts
    LSE by that constant; a bias broadcast over batch and heads equals its
    materialised copy."""
    B, H, S, D = 2, 3, 8, 4
    q, k, v, _ = _tiny(seed, B=B, H=H, Hkv=1, S=S, D=D)
    slopes = [0.25, 0.5, 1.25]
    i = np.arange(S)
    alibi = np.stack([-sl * (i[:, None] - i[None, :]) for sl in slopes])[None].astype(np.float64)
    a = oracle.attention_forward(q, k, v, rope="neox", mask="causal", alibi_slopes=slopes, scale=0.7)
    b = oracle.attention_forward(q, k, v, rope="neox", mask="causal", bias=alibi, scale=0.7)
    assert np.allclose(a[0], b[0], atol=TOL, rtol=0) and np.allclose(a[1], b[1], atol=TOL, rtol=0)
    upper = np.where(i[None, :] > i[:, None], -np.inf, 0.0)
    a = oracle.attention_forward(q, k, v, rope="interleaved", mask="causal")
    b = oracle.attention_forward(q, k, v, rope="interleaved", mask="none", bias=upper)
    assert np.allclose(a[0], b[0], atol=TOL, rtol=0) and np.allclose(a[1], b[1], atol=TOL, rtol=0)
    c = _rng(seed).standard_normal((B, H, S, 1)) * 3.0
    a = oracle.attention_forward(q, k, v, mask="none", scale=0.9)
    b = oracle.attention_forward(q, k, v, mask="none", scale=0.9, bias=np.broadcast_to(c, (B, H, S, S)))
    assert np.allclose(a[0], b[0], atol=1e-12, rtol=0)
    assert np.allclose(b[1] - a[1], c[..., 0], atol=1e-12, rtol=0)
    one = _bias(seed, 1, 1, S)
    a = oracle.attention_forward(q, k, v, mask="none", bias=one)
    b = oracle.attention_forward(q, k, v, mask="none", bias=np.broadcast_to(one, (B, H, S, S)).copy())
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def check_relu_closed_forms(seed=42):
    """Relu attention: causal row 0 is max(s_00, 0) v_0; scores all below zero
    give O = 0; O is positively homogeneous in the scale (max(a s, 0) =
    a max(s, 0)) and linear in V."""
    q, k, v, _ = _tiny(seed, B=1, H=2, Hkv=1, S=6, D=4)
    O, L = oracle.attention_forward(q, k, v, rope="neox", mask="causal", norm="relu", scale=0.8)
    assert L is None
    s00 = 0.8 * q[0, :, 0] @ k[0, 0, 0]                     # RoPE is the identity at position 0
    assert np.allclose(O[0, :, 0], np.maximum(s00, 0.0)[:, None] * v[0, 0, 0][None, :], atol=TOL, rtol=0)
    neg = np.full((1, 2, 6, 6), -1e3)
    O, _ = oracle.attention_forward(q, k, v, mask="none", norm="relu", bias=neg)
    assert (O == 0).all()
    a, _ = oracle.attention_forward(q, k, v, mask="sliding_window", window=3, norm="relu", scale=0.5)
    b, _ = oracle.attention_forward(q, k, v, mask="sliding_window", window=3, norm="relu", scale=1.5)
    assert np.allclose(3.0 * a, b, atol=TOL, rtol=0)
    c, _ = oracle.attention_forward(q, k, -2.0 * v, mask="sliding_window", window=3, norm="relu", scale=0.5)
    assert np.allclose(-2.0 * a, c, atol=TOL, rtol=0)


def check_bias_relu_backward_fd(norm, seed=43):
    """Gradients with a bias tensor (softmax or relu) against central finite
    differences of the brute force; relu kinks (s = 0) are measure-zero for
    these random inputs."""
    q, k, v, do = _tiny(seed, B=1, H=2, Hkv=1, S=5, D=4)
    bias = _bias(seed, 1, 2, 5)
    kw = dict(rope="neox", theta=10000.0, mask="causal", window=None, alibi_slopes=None, scale=0.6)
    dq, dk, dv = oracle.attention_backward(q, k, v, do, bias=bias, norm=norm, **kw)
    ql, kl, vl, dol = q.tolist(), k.tolist(), v.tolist(), do.tolist()
    bl = bias.tolist()

    def f():
        return bruteforce.loss(ql, kl, vl, dol, bias=bl, norm=norm, **kw)

    assert np.allclose(dq, np.array(bruteforce.finite_difference_grad(ql, f)), atol=1e-7)
    assert np.allclose(dk, np.array(bruteforce.finite_difference_grad(kl, f)), atol=1e-7)
    assert np.allclose(dv, np.array(bruteforce.finite_difference_grad(vl, f)), atol=1e-7)


def check_relu_gate_precision(seed=44):
    """The fp16 relu gate equals the exact one when the rotated operands are
    representable in fp16 (small integers, no RoPE), and differs exactly where
    rounding to fp16 moves a score across zero (a constructed case)."""
    r = _rng(seed)
    q = r.integers(-3, 4, (1, 2, 6, 4)).astype(np.float64)
    k = r.integers(-3, 4, (1, 1, 6, 4)).astype(np.float64)
    v, do = r.standard_normal((1, 1, 6, 4)), r.standard_normal((1, 2, 6, 4))
    kw = dict(mask="none", norm="relu", scale=0.5)
    a = oracle.attention_backward(q, k, v, do, relu_gate="exact", **kw)
    b = oracle.attention_backward(q, k, v, do, relu_gate="fp16", **kw)
    assert all(np.array_equal(x, y) for x, y in zip(a, b))
    # one query, two keys; q.k1 = 1e-4 exactly in fp64 but 0 after fp16 rounding of q
    q = np.zeros((1, 1, 1, 2)); q[0, 0, 0] = [1.0 + 2.0 ** -13, 1.0]
    k = np.zeros((1, 1, 1, 2)); k[0, 0, 0] = [1.0, -1.0]
    v = np.ones((1, 1, 1, 2)); do = np.ones((1, 1, 1, 2))
    ex = oracle.attention_backward(q, k, v, do, mask="none", norm="relu", scale=1.0, relu_gate="exact")
    hf = oracle.attention_backward(q, k, v, do, mask="none", norm="relu", scale=1.0, relu_gate="fp16")
    assert np.allclose(ex[0][0, 0, 0], 2.0 * k[0, 0, 0])        # s = 2^-13 > 0: dS = dP = 2
    assert np.array_equal(hf[0], np.zeros_like(hf[0]))          # fp16 q.k = 0: gate closed


def check_backward_given_output(seed=45):
    """delta from a given forward output: with the exact O the gradients are
    the default ones; with O + E every row of dS sums to -rowsum(dO * E)
    (the softmax rows sum to 1, so sum_j dS_ij = sum_j P_ij dP_ij - delta_i),
    where the definitional delta makes every row sum to zero."""
    r = _rng(seed)
    q, k, v = r.standard_normal((1, 2, 9, 4)), r.standard_normal((1, 1, 9, 4)), r.standard_normal((1, 1, 9, 4))
    do = r.standard_normal((1, 2, 9, 4))
    kw = dict(rope="neox", mask="causal")
    O, _ = oracle.attention_forward(q, k, v, **kw)
    a = oracle.attention_backward(q, k, v, do, **kw)
    b = oracle.attention_backward(q, k, v, do, o=O, **kw)
    assert all(np.allclose(x, y, rtol=0, atol=1e-12) for x, y in zip(a, b))
    E = 0.01 * r.standard_normal(O.shape)
    *_, inter = oracle.attention_backward(q, k, v, do, o=O + E, return_intermediates=True, **kw)
    for h in range(2):
        expect = -np.sum(do[0, h] * E[0, h], axis=1)
        assert np.allclose(inter["dS"][(0, h)].sum(axis=1), expect, rtol=0, atol=1e-12)
