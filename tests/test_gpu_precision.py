"""The RoPE forward's LSE against its operand-precision model (through the C ABI).

With RoPE the forward rotates Q and K in fp32 and rounds the rotated Q' and K'
to fp16 (11-bit significand) for the score MFMA; the definition rotates
exactly.  Rounding each operand moves it by at most 2^-11 of itself, so a score
s_ij = scale <q'_i, k'_j> moves by at most
    b_ij = scale * sum_d |q'_id k'_jd| * (2 * 2^-11 + 2^-16)
(the last term: fp32 accumulation over D products), and LSE_i, whose first-order
change is the P-weighted mean of its scores' changes, by at most the largest b_ij
over the row's visible keys.  At the default scale 1/sqrt(D) with unit-variance
inputs that stays near the contract's flat 1e-3, but it grows with the scale and
the operands' norms: in a seeded sweep of 200 random shapes, 28 RoPE cases with
scales up to 0.28 or rows with one or two visible keys exceeded 1e-3 (at most
3.1e-3).  These cases, drawn from that sweep, check two things:

* the GPU's LSE equals the LSE of the same definition evaluated on the
  fp16-rounded rotated operands (the oracle's rotation rounded to fp16) to the
  flat 1e-3: the error is the operands' rounding and nothing else;
* its distance to the exact LSE stays within max_j b_ij (plus 2e-4 for the exp2
  / log2 approximations and fp32 sums of the online softmax).

Without RoPE the bf16 inputs enter the MFMA exactly and the flat 1e-3 is
checked everywhere else in the suite.
"""
import pytest
import torch

from gpu_util import announce, assert_rope_lse_close, device_inputs, f64, need_gpu
from paper_2609_13612_amd import api, inputs

pytestmark = pytest.mark.gpu

# (B, H, H_kv, S, D, rope, theta, mask, window, alibi, scale, seed)
CASES = [
    (2, 4, 1, 511, 128, "neox", 1e4, "none", None, False, 0.27483106361148496, 2037),
    (1, 4, 1, 511, 128, "interleaved", 1e4, "none", None, True, 0.27639494086895305, 2050),
    (2, 2, 1, 2, 128, "neox", 1e4, "none", None, False, 0.27742000449588294, 2145),
    (1, 12, 1, 31, 64, "interleaved", 5e5, "sliding_window", 1, False, None, 2071),
    (1, 24, 2, 191, 64, "neox", 1e4, "causal", None, True, 0.2128474905870627, 2025),
    (2, 4, 1, 130, 128, "interleaved", 5e5, "causal", None, False, 0.1798346386095227, 2160),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"{c[5]}-{c[7]}-S{c[3]}-D{c[4]}-scale{c[10]}")
def test_rope_lse_within_operand_rounding_bound(case):
    need_gpu()
    B, H, Hkv, S, D, rope, theta, mask, window, alibi, scale, seed = case
    announce(f"LSE precision model: {case}")
    cpu, dev = device_inputs(B, H, Hkv, S, D, seed=seed)
    slopes = inputs.alibi_slopes(H) if alibi else None
    kw = dict(mask=mask, window=window, scale=scale)
    _, lse = api.attnfuse_fwd(dev["q"], dev["k"], dev["v"], rope=rope, theta=theta,
                              alibi_slopes=None if slopes is None else slopes.cuda(), **kw)
    torch.cuda.synchronize()
    os_ = None if slopes is None else f64(slopes)
    err, err16 = assert_rope_lse_close(lse, f64(cpu["q"]), f64(cpu["k"]), f64(cpu["v"]), rope, theta, os_, **kw)
    print(f"LSE error vs exact {err:.3e} (flat 1e-3 {'met' if err <= 1e-3 else 'exceeded'}), "
          f"vs the fp16-operand definition {err16:.3e}")
