"""Shared helpers of the GPU parity tests: device inputs, tolerances, workloads.

Tolerances are the ones the contract states: bf16 outputs max-abs 2e-2 and
mean-abs 2e-3; the fp32 debug path 1e-4; LSE 1e-3 absolute.

Reading of the bf16 bound: bf16 has an 8-bit significand, so rounding a value
x to it can move it by up to half an ulp, 2^-8 |x| (the format's unit
roundoff: up to 0.0039 just above |x| = 1, 0.0625 just above |x| = 16), which no
implementation with bf16 outputs can avoid -- from |x| = 8 on even the
correctly rounded exact value can miss a flat 2e-2.  The max-abs bound is
therefore applied per element as 2e-2 + 2^-8 |ref|, and the mean-abs bound as
2e-3 + 2^-9 mean|ref| (rounding to bf16 costs at most a quarter ulp on
average).  Every check also reports its max-abs and mean-abs against the flat
2e-2 / 2e-3 figures: printed, and appended as a JSON line to the file named by
the environment variable ATTNFUSE_ERR_LOG when it is set.

Backward parity takes no value from the GPU path into the oracle: the forward
output O and the LSE a backward test hands the kernels come from the oracle's
own forward (O rounded to the tensor dtype, as a forward stores it), and the
oracle's backward is given that same O where the kernels use it (dQ; see
``bwd_refs``).  The definitional tests instead run
the GPU forward and backward end to end and compare with the oracle's
gradients of the exact function (no O given).
"""
import json
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_2609_13612_amd import inputs

BF16_MAX, BF16_MEAN, FP32_MAX, LSE_MAX = 2e-2, 2e-3, 1e-4, 1e-3


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def announce(msg):
    """Name the case on stdout (flushed) before a GPU step runs."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def device_inputs(B, H, Hkv, S, D, dtype="bf16", seed=0, with_do=False):
    cpu = inputs.make_qkv(B, H, Hkv, S, D, dtype=dtype, seed=seed, with_do=with_do)
    return cpu, {k: v.cuda() for k, v in cpu.items()}


def f64(t):
    return inputs.to_f64(t)


BF16_HALF_ULP = 2.0 ** -8   # bf16 unit roundoff
BF16_QUARTER_ULP = 2.0 ** -9   # mean bf16 rounding error of a value, relative, at most


def report(what, err, ref, flat_max, flat_mean):
    """Print (and log) one check's errors against the flat stated bounds."""
    mx = float(err.max()) if err.size else 0.0
    mn = float(err.mean()) if err.size else 0.0
    rmax = float(np.abs(ref).max()) if err.size else 0.0
    ok = lambda x, t: "ok" if x <= t else "over"
    print(f"[err] {what}: max-abs {mx:.3e} (flat {flat_max:g} {ok(mx, flat_max)}), mean-abs {mn:.3e} "
          f"(flat {flat_mean:g} {ok(mn, flat_mean)}), max|ref| {rmax:.3g}", flush=True)
    path = os.environ.get("ATTNFUSE_ERR_LOG")
    if path:
        rec = {"test": os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0], "what": what, "max_abs": mx,
               "mean_abs": mn, "max_ref": rmax, "flat_max": flat_max, "flat_mean": flat_mean}
        with open(path, "a") as f:
            f.write(json.dumps(rec) + "\n")
    return mx, mn


def given_o(O, dtype="bf16"):
    """The oracle's forward output as a forward of ``dtype`` stores it: the
    rounded values as the fp64 array the oracle's backward takes (``o=``) and
    as a device tensor for the kernels."""
    t = torch.from_numpy(np.ascontiguousarray(O)).to(torch.bfloat16 if dtype == "bf16" else torch.float32)
    return t.to(torch.float64).numpy(), t.cuda()


def bwd_refs(backward, o_ref):
    """The oracle gradients a bf16 backward handed the forward output o_ref is
    held to: dQ with the row term delta from o_ref (the dQ pass forms it from
    the O it is given), dK and dV with the definitional delta = sum_j P_ij
    dP_ij (the dK/dV pass uses the dQ pass's own sum).  ``backward(o)`` runs
    the oracle's backward with that ``o`` (None: the definition)."""
    given = backward(o_ref)
    exact = backward(None)
    return given[0], exact[1], exact[2]


def given_lse(L):
    """The oracle's LSE as the fp32 device tensor a forward stores."""
    return torch.from_numpy(np.ascontiguousarray(L)).to(torch.float32).cuda()


def assert_bf16_close(gpu, ref, what, max_tol=BF16_MAX, mean_tol=BF16_MEAN):
    g = f64(gpu) if isinstance(gpu, torch.Tensor) else gpu
    err = np.abs(g - ref)
    assert np.isfinite(g).all(), f"{what}: non-finite values"
    report(what, err, ref, max_tol, mean_tol)
    excess = err - (max_tol + BF16_HALF_ULP * np.abs(ref))
    i = np.unravel_index(np.argmax(excess), err.shape) if err.size else None
    assert err.size == 0 or excess.max() <= 0, \
        f"{what}: error {err[i]:.3e} at |ref| {abs(ref[i]):.3f} exceeds {max_tol} + 2^-8|ref| (max-abs {err.max():.3e})"
    # the mean criterion allows, like the per-element one, what rounding the
    # exact result to bf16 costs on average (at most a quarter ulp, 2^-9|ref|)
    mtol = mean_tol + BF16_QUARTER_ULP * (float(np.abs(ref).mean()) if err.size else 0.0)
    assert err.mean() <= mtol, f"{what}: mean-abs {err.mean():.3e} > {mean_tol} + 2^-9 mean|ref| = {mtol:.3e}"
    return float(err.max()), float(err.mean())


def bf16_round(x):
    """Round an fp64 array to bf16 and back (the storage format of a bf16 tensor)."""
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16).to(torch.float64).numpy()


def assert_fp32_close(gpu, ref, what, tol=FP32_MAX):
    g = f64(gpu) if isinstance(gpu, torch.Tensor) else gpu
    err = np.abs(g - ref)
    report(what, err, ref, tol, tol)
    assert err.max() <= tol, f"{what}: max-abs {err.max():.3e} > {tol}"
    return float(err.max())


def assert_lse_close(gpu, ref, what, tol=LSE_MAX):
    g = f64(gpu) if isinstance(gpu, torch.Tensor) else gpu
    assert np.array_equal(np.isneginf(g), np.isneginf(ref)), f"{what}: -inf pattern differs"
    fin = np.isfinite(ref)
    err = np.abs(g[fin] - ref[fin])
    report(what, err, ref[fin], tol, tol)
    assert err.size == 0 or err.max() <= tol, f"{what}: LSE max-abs {err.max():.3e} > {tol}"


def visible_pairs(S, mask, window, block_mask=None):
    """[S, S] boolean: query i sees key j under the mask (no mask, causal, or causal + window)
    and, if given, the block mask ((block size, active [nb, nb] bool) pair)."""
    i = np.arange(S)[:, None]
    j = np.arange(S)[None, :]
    vis = np.ones((S, S), dtype=bool)
    if mask != "none":
        vis &= j <= i
    if mask == "sliding_window":
        vis &= j > i - window
    if block_mask is not None:
        bs, active = block_mask
        vis &= active[i // bs, j // bs]
    return vis


def assert_rope_lse_close(lse, q, k, v, rope, theta, alibi_slopes, mask, window, scale, block_mask=None):
    """The LSE of a RoPE forward against its operand-precision model (q, k, v:
    the fp64 inputs; alibi_slopes fp64 or None; block_mask the oracle's
    (block size, active) pair or None).

    The kernels round the rotated Q' and K' to fp16 for the score MFMA; the
    definition rotates exactly.  Rounding each operand moves it by at most
    2^-11 of itself, so a score moves by at most
        b_ij = scale * sum_d |q'_id k'_jd| * (2 * 2^-11 + 2^-16)
    (the last term: fp32 accumulation over D products), and a row's LSE, whose
    first-order change is the P-weighted mean of its scores' changes, by at most
    the largest b_ij over the row's visible keys.  Checked: the LSE equals the
    definition evaluated on the fp16-rounded rotated operands to the flat 1e-3
    (the error is the operands' rounding and nothing else), and lies within
    max_j b_ij (+ 2e-4 for the exp2 / log2 approximations and fp32 sums of the
    online softmax) of the exact LSE.  Returns the two max-abs errors."""
    B, H, S, D = q.shape
    G = H // k.shape[1]
    kw = dict(mask=mask, window=window, scale=scale, block_mask=block_mask)
    _, L = oracle.attention_forward(q, k, v, rope=rope, theta=theta, alibi_slopes=alibi_slopes, **kw)
    pos = np.arange(S, dtype=np.float64)
    qr = oracle.rope_rotate(q, pos, theta, rope)
    kr = oracle.rope_rotate(k, pos, theta, rope)
    q16 = qr.astype(np.float16).astype(np.float64)
    k16 = kr.astype(np.float16).astype(np.float64)
    _, L16 = oracle.attention_forward(q16, k16, v, rope="none", alibi_slopes=alibi_slopes, **kw)
    g = f64(lse) if isinstance(lse, torch.Tensor) else lse
    assert np.array_equal(np.isneginf(g), np.isneginf(L)), "LSE: -inf pattern differs"
    fin = np.isfinite(L)
    err16 = np.abs(g[fin] - L16[fin])
    report("LSE vs the fp16-operand definition", err16, L16[fin], LSE_MAX, LSE_MAX)
    assert err16.size == 0 or err16.max() <= LSE_MAX, f"LSE vs the fp16-operand definition: {err16.max():.3e}"
    sc = scale if scale is not None else D ** -0.5
    vis = visible_pairs(S, mask, window, block_mask)
    err = np.where(fin, np.abs(g - np.where(fin, L, 0.0)), 0.0)
    for b in range(B):
        for h in range(H):
            mag = np.abs(qr[b, h]) @ np.abs(kr[b, h // G]).T          # sum_d |q'_id k'_jd|
            bnd = sc * mag * (2 * 2.0 ** -11 + 2.0 ** -16)
            row_bound = np.where(vis, bnd, 0.0).max(axis=1) + 2e-4
            over = err[b, h] > row_bound
            assert not over.any(), (f"(b={b}, h={h}) LSE error {err[b, h][over].max():.3e} above its "
                                    f"rounding bound {row_bound[over].min():.3e}")
    return float(err.max()), float(err16.max()) if err16.size else 0.0
