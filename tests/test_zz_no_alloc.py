"""attnfuse_decode_noalloc (the decode entry point that allocates nothing)
against attnfuse_decode, through the C ABI: the same kernels with the
partials in the library's static scratch instead of a caller's workspace, so
the outputs must be identical bit for bit.  Two calls in a row, the second
with a smaller problem (the scratch keeps the first call's contents), then a
request larger than the scratch."""

import pytest
import torch

from gpu_util import announce, need_gpu
from paper_2609_13612_amd import api, inputs

pytestmark = pytest.mark.gpu

CASES = [
    # B, H, H_kv, S_kv, D, rope, mask, window, ragged lengths
    (2, 32, 8, 4096, 128, "neox", "causal", None, [4096, 2500]),
    (1, 8, 2, 700, 64, "interleaved", "sliding_window", 300, None),
]


def test_decode_noalloc_matches_workspace_entry_point():
    need_gpu()
    for i, (B, H, Hkv, S, D, rope, mask, window, lens) in enumerate(CASES):
        announce(f"decode noalloc call {i}: B={B} H={H} Hkv={Hkv} S={S} D={D} rope={rope} mask={mask}")
        c = inputs.make_decode(B, H, Hkv, S, D, seed=200 + i)
        q, k, v = c["q"].cuda(), c["k"].cuda(), c["v"].cuda()
        cl = None if lens is None else torch.tensor(lens, dtype=torch.int32, device="cuda")
        kw = dict(rope=rope, theta=500000.0, mask=mask, window=window)
        o_ws, lse_ws = api.attnfuse_decode(q, k, v, cl, **kw)
        o_na, lse_na = api.attnfuse_decode_noalloc(q, k, v, cl, **kw)
        torch.cuda.synchronize()
        assert torch.equal(o_na, o_ws), f"call {i}: O differs"
        assert torch.equal(lse_na, lse_ws), f"call {i}: LSE differs"


def test_decode_noalloc_rejects_requests_beyond_the_scratch():
    need_gpu()
    B, H, Hkv, S, D = 1, 32, 1, 1 << 20, 128
    assert api.attnfuse_decode_workspace_bytes(B, H, Hkv, S, D) > 32 << 20
    q = torch.zeros(B, H, D, dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros(B, Hkv, S, D, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(api.AttnFuseError) as e:
        api.attnfuse_decode_noalloc(q, kc, kc.clone())
    assert e.value.code == -4
