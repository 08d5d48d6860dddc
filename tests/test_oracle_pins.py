"""The fp64 oracle against closed forms, invariants, brute force and library routines (CPU)."""
import pytest

import oracle_pins as P

ROPES = ["neox", "interleaved"]


def test_frequencies():
    P.check_frequencies()


@pytest.mark.parametrize("kind", ROPES)
def test_rope_d2_closed_form(kind):
    P.check_rope_d2_closed_form(kind)


@pytest.mark.parametrize("kind", ROPES)
def test_rope_pairing(kind):
    P.check_rope_pairing(kind)


@pytest.mark.parametrize("kind", ROPES)
def test_rope_preserves_norms(kind):
    P.check_rope_norm(kind)


@pytest.mark.parametrize("kind", ROPES)
def test_rope_dot_depends_on_relative_position(kind):
    P.check_rope_relative(kind)


@pytest.mark.parametrize("kind", ROPES)
def test_rope_inverse_and_identity(kind):
    P.check_rope_inverse(kind)


@pytest.mark.parametrize("kind", ROPES)
def test_rope_vs_givens_matrix(kind):
    P.check_rope_vs_givens(kind)


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_forward_vs_bruteforce(variant):
    P.check_forward_vs_bruteforce(variant)


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_softmax_rows_sum_to_one(variant):
    P.check_softmax_rows(variant)


@pytest.mark.parametrize("kind", ["none"] + ROPES)
def test_causal_first_rows_closed_form(kind):
    P.check_causal_first_rows(kind)


@pytest.mark.parametrize("kind", ["none"] + ROPES)
def test_window_one_gives_v(kind):
    P.check_window_one(kind)


def test_window_reductions():
    P.check_window_reductions()


def test_alibi_special_cases():
    P.check_alibi_special_cases()


@pytest.mark.parametrize("mask", ["none", "causal"])
def test_vs_torch_sdpa(mask):
    P.check_vs_torch_sdpa(mask)


@pytest.mark.parametrize("kind", ROPES)
@pytest.mark.parametrize("mask", ["none", "causal", "sliding_window"])
def test_position_shift_invariance(kind, mask):
    P.check_position_shift(kind, mask)


def test_gqa_equals_repeat_kv():
    P.check_gqa_repeat_kv()


def test_sampled_rows_match_full():
    P.check_rows_match_full()


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_backward_finite_differences(variant):
    P.check_backward_fd(variant)


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_backward_vs_torch_autograd(variant):
    P.check_backward_vs_torch_autograd(variant)


def test_backward_identities():
    P.check_backward_identities()


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_decode_vs_bruteforce(variant):
    P.check_decode_vs_bruteforce(variant)


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_decode_is_last_prefill_row(variant):
    P.check_decode_is_last_prefill_row(variant)


@pytest.mark.parametrize("kind", ["none"] + ROPES)
def test_decode_closed_forms(kind):
    P.check_decode_closed_forms(kind)


def test_decode_ignores_stale_entries():
    P.check_decode_ignores_stale_entries()


@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_block_mask_vs_bruteforce(variant):
    P.check_block_mask_vs_bruteforce(variant)


def test_block_mask_reductions():
    P.check_block_mask_reductions()


def test_block_mask_backward_fd():
    P.check_block_mask_backward_fd()


@pytest.mark.parametrize("norm", ["softmax", "relu"])
@pytest.mark.parametrize("variant", P.VARIANTS, ids=lambda v: "-".join(map(str, v)))
def test_bias_relu_vs_bruteforce(variant, norm):
    P.check_bias_relu_vs_bruteforce(variant, norm)


def test_bias_reductions():
    P.check_bias_reductions()


def test_relu_closed_forms():
    P.check_relu_closed_forms()


@pytest.mark.parametrize("norm", ["softmax", "relu"])
def test_bias_relu_backward_fd(norm):
    P.check_bias_relu_backward_fd(norm)


def test_relu_gate_precision():
    P.check_relu_gate_precision()


def test_backward_given_output():
    P.check_backward_given_output()
