"""Plant plausible mistakes in the oracle (on the CPU) and check that some pin catches each.

This shows the pins in oracle_pins.py are discriminating: a dropped term, a
wrong sign or index, or a transposed operand anywhere in the oracle fails at
least one of them.
"""
import numpy as np
import pytest

import oracle
import oracle.attention as oatt
import oracle.decode as odec
import oracle.rope as orope
import oracle_pins as P

FWD = ("neox", "causal", None, False)
ALIBI = ("neox", "causal", None, True)
SW = ("neox", "sliding_window", 3, False)


def _fails(checks):
    for check in checks:
        try:
            check()
        except AssertionError:
            return True
    return False


def _wrong_sign_rotate(x, positions, theta, kind, inverse=False):
    return _REAL_ROTATE(x, positions, theta, kind, inverse=not inverse)


def _no_inverse_rotate(x, positions, theta, kind, inverse=False):
    return _REAL_ROTATE(x, positions, theta, kind, inverse=False)


_REAL_ROTATE = orope.rope_rotate


def _bad_pairs(D, kind):
    half = D // 2
    i = np.arange(half)
    if kind == "neox":                       # reversed partner: (i, D-1-i)
        return i, D - 1 - i
    return 2 * i, 2 * i + 1


def _bad_freq(D, theta):
    i = np.arange(D // 2, dtype=np.float64)
    return np.power(np.float64(theta), -1.0 * i / D)   # dropped factor 2


def _bad_kv_head(h, H, Hkv):
    return h % Hkv                           # interleaved instead of contiguous groups


def _bad_alibi(slope, rows, cols):
    return slope * (np.asarray(rows)[:, None] - np.asarray(cols)[None, :]).astype(np.float64)


def _bad_visibility(i, j, mask, window=None, block_mask=None):
    i2 = np.asarray(i)[:, None]
    j2 = np.asarray(j)[None, :]
    if mask == "sliding_window":
        return (j2 <= i2) & (j2 >= i2 - window)   # W + 1 keys
    return _REAL_VIS(i, j, mask, window, block_mask)


def _transposed_blocks(i, j, block_mask):
    bs, active = block_mask
    active = np.asarray(active, dtype=bool)
    return active.T[np.asarray(i)[:, None] // bs, np.asarray(j)[None, :] // bs]


_REAL_VIS = oatt.visibility


def _no_scale_defaults(D, scale, alibi_slopes, H):
    sc, slopes = _REAL_DEFAULTS(D, scale, alibi_slopes, H)
    return 1.0, slopes


_REAL_DEFAULTS = oatt._defaults


def _bad_decode_visible(j, p, mask, window=None):
    j = np.asarray(j)
    if mask == "sliding_window":
        return (j <= p) & (j >= p - window)        # W + 1 keys
    return j <= p


_REAL_BIAS_OF = oatt._bias_of


def _scaled_bias_of(bias, B, H, S):
    b = _REAL_BIAS_OF(bias, B, H, S)
    return None if b is None else 0.41 * b          # the softmax scale applied to the bias too


def _transposed_bias_of(bias, B, H, S):
    b = _REAL_BIAS_OF(bias, B, H, S)
    return None if b is None else np.swapaxes(b, -1, -2)


def _normalised_relu(s):
    r = np.maximum(s, 0.0)
    tot = r.sum(axis=1, keepdims=True)
    return r / np.where(tot > 0, tot, 1.0)


MUTATIONS = {
    "rotation_sign": [(oatt, "rope_rotate", _wrong_sign_rotate), (orope, "rope_rotate", _wrong_sign_rotate),
                      (oracle, "rope_rotate", _wrong_sign_rotate)],
    "decode_rotation_sign": [(odec, "rope_rotate", _wrong_sign_rotate)],
    "decode_gqa_mapping": [(odec, "kv_head", _bad_kv_head)],
    "decode_query_position": [(odec, "query_position", lambda n: n)],   # one past the newest token
    "decode_window_boundary": [(odec, "decode_visible", _bad_decode_visible)],
    "neox_partner": [(orope, "rope_pair_indices", _bad_pairs)],
    "frequency_exponent": [(orope, "rope_frequencies", _bad_freq), (oracle, "rope_frequencies", _bad_freq)],
    "gqa_mapping": [(oatt, "kv_head", _bad_kv_head)],
    "alibi_sign": [(oatt, "alibi_bias", _bad_alibi)],
    "window_boundary": [(oatt, "visibility", _bad_visibility)],
    "block_mask_transposed": [(oatt, "block_visible", _transposed_blocks)],
    "dropped_scale": [(oatt, "_defaults", _no_scale_defaults)],
    "gradient_not_unrotated": [(oatt, "rope_rotate", _no_inverse_rotate)],
    "bias_scaled": [(oatt, "_bias_of", _scaled_bias_of)],
    "bias_transposed": [(oatt, "_bias_of", _transposed_bias_of)],
    "relu_normalised": [(oatt, "_relu_rows", _normalised_relu)],
    "relu_gradient_unmasked": [(oatt, "_relu_grad", lambda s, dP: dP)],
    "given_output_ignored": [(oatt, "_row_delta", lambda P_, dP, dO_rows, o_rows: np.sum(P_ * dP, axis=1))],
}

CHECKS = [
    P.check_frequencies,
    lambda: P.check_rope_vs_givens("neox"),
    lambda: P.check_rope_d2_closed_form("neox"),
    lambda: P.check_forward_vs_bruteforce(FWD),
    lambda: P.check_forward_vs_bruteforce(ALIBI),
    lambda: P.check_forward_vs_bruteforce(SW),
    lambda: P.check_window_one("neox"),
    P.check_gqa_repeat_kv,
    P.check_alibi_special_cases,
    lambda: P.check_backward_fd(FWD),
    lambda: P.check_decode_vs_bruteforce(FWD),
    lambda: P.check_decode_vs_bruteforce(ALIBI),
    lambda: P.check_decode_vs_bruteforce(SW),
    lambda: P.check_decode_closed_forms("neox"),
    lambda: P.check_block_mask_vs_bruteforce(FWD),
    lambda: P.check_bias_relu_vs_bruteforce(FWD, "softmax"),
    lambda: P.check_bias_relu_vs_bruteforce(FWD, "relu"),
    P.check_bias_reductions,
    P.check_relu_closed_forms,
    lambda: P.check_bias_relu_backward_fd("relu"),
    P.check_backward_given_output,
]


def test_pins_pass_unmutated():
    assert not _fails(CHECKS)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    for module, attr, fake in MUTATIONS[name]:
        monkeypatch.setattr(module, attr, fake)
    assert _fails(CHECKS), f"no pin caught the planted mistake {name!r}"
