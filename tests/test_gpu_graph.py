"""HIP-graph capture of the entry points through the C ABI.

The library allocates nothing, synchronises nothing and issues no memset (the
RoPE cos/sin table is the caller's), so every entry point can be captured,
the first call included: the fused forward and backward (also with a dense
bias or relu attention), the block-sparse forward and backward, decode and
the separate path (rotation kernel, then the forward without RoPE), and a
RoPE call whose table the binding has not built yet (its fill kernel is
captured with it).  Each test captures once, then replays on three fresh inputs
copied into the captured buffers, with eager calls and synchronisations in
between, and checks every replay bit for bit against the eager result on the
same inputs (the kernels use no atomics, so they are deterministic).
"""
import pytest
import torch

from gpu_util import announce, device_inputs, need_gpu
from paper_2609_13612_amd import api, blockmask, inputs

pytestmark = pytest.mark.gpu

SEEDS = (71, 72, 73)


def _capture(fn):
    g = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def test_graph_fwd_bwd_replays():
    """Fused RoPE + causal forward then backward, GQA, S = 1000 (ragged tail)."""
    need_gpu()
    announce("graph capture: fwd + bwd")
    B, H, Hkv, S, D = 1, 8, 2, 1000, 128
    kw = dict(rope="neox", theta=500000.0, mask="causal")
    _, d0 = device_inputs(B, H, Hkv, S, D, seed=70, with_do=True)
    q, k, v, do = (d0[n].clone() for n in ("q", "k", "v", "do"))
    o, lse = api.attnfuse_fwd(q, k, v, **kw)            # eager warm-up
    api.attnfuse_bwd(q, k, v, o, do, lse, **kw)
    o_s, lse_s = torch.empty_like(q), torch.empty(B, H, S, device="cuda")
    dq_s, dk_s, dv_s = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(api.attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, "neox"), device="cuda", dtype=torch.uint8)

    def step():
        api.attnfuse_fwd(q, k, v, out=o_s, lse=lse_s, **kw)
        api.attnfuse_bwd(q, k, v, o_s, do, lse_s, dq=dq_s, dk=dk_s, dv=dv_s, workspace=ws, **kw)

    g = _capture(step)
    for seed in SEEDS:
        _, d = device_inputs(B, H, Hkv, S, D, seed=seed, with_do=True)
        o_e, lse_e = api.attnfuse_fwd(d["q"], d["k"], d["v"], **kw)
        grads_e = api.attnfuse_bwd(d["q"], d["k"], d["v"], o_e, d["do"], lse_e, **kw)
        torch.cuda.synchronize()
        for dst, name in ((q, "q"), (k, "k"), (v, "v"), (do, "do")):
            dst.copy_(d[name])
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_s, o_e) and torch.equal(lse_s, lse_e), f"seed {seed}: forward replay differs"
        for name, a, b in zip(("dQ", "dK", "dV"), (dq_s, dk_s, dv_s), grads_e):
            assert torch.equal(a, b), f"seed {seed}: {name} replay differs"


def test_graph_cold_first_call_replays():
    """The first call for a (D, theta) captured with nothing built before it:
    the binding fills a fresh cos/sin table inside the capture, the forward and
    backward read it, and the replays match eager calls (made afterwards)."""
    need_gpu()
    announce("graph capture: cold first RoPE call")
    B, H, Hkv, S, D = 1, 4, 2, 700, 64
    theta = 123457.0                                      # no other test builds this table
    assert not any(key[1:] == (D, float(theta)) for key in api._TABLES)
    kw = dict(rope="neox", theta=theta, mask="sliding_window", window=200)
    _, d0 = device_inputs(B, H, Hkv, S, D, seed=70, with_do=True)
    q, k, v, do = (d0[n].clone() for n in ("q", "k", "v", "do"))
    o_s, lse_s = torch.empty_like(q), torch.empty(B, H, S, device="cuda")
    dq_s, dk_s, dv_s = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(api.attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, "neox"), device="cuda", dtype=torch.uint8)

    def step():
        api.attnfuse_fwd(q, k, v, out=o_s, lse=lse_s, **kw)
        api.attnfuse_bwd(q, k, v, o_s, do, lse_s, dq=dq_s, dk=dk_s, dv=dv_s, workspace=ws, **kw)

    g = _capture(step)
    for seed in SEEDS:
        _, d = device_inputs(B, H, Hkv, S, D, seed=seed, with_do=True)
        for dst, name in ((q, "q"), (k, "k"), (v, "v"), (do, "do")):
            dst.copy_(d[name])
        g.replay()
        torch.cuda.synchronize()
        o_e, lse_e = api.attnfuse_fwd(d["q"], d["k"], d["v"], **kw)
        grads_e = api.attnfuse_bwd(d["q"], d["k"], d["v"], o_e, d["do"], lse_e, **kw)
        torch.cuda.synchronize()
        assert torch.equal(o_s, o_e) and torch.equal(lse_s, lse_e), f"seed {seed}: forward replay differs"
        for name, a, b in zip(("dQ", "dK", "dV"), (dq_s, dk_s, dv_s), grads_e):
            assert torch.equal(a, b), f"seed {seed}: {name} replay differs"


def test_graph_blocksparse_replays():
    """Block-sparse forward then backward over a BigBird-style mask, D = 64,
    S = 1024, with RoPE."""
    need_gpu()
    announce("graph capture: block-sparse fwd + bwd")
    B, H, Hkv, S, D = 2, 4, 4, 1024, 64
    kw = dict(rope="neox")
    bm = blockmask.block_mask_from_dense(torch.from_numpy(inputs.bigbird_blocks(S // 64, seed=3)), S, device="cuda")
    _, d0 = device_inputs(B, H, Hkv, S, D, seed=70, with_do=True)
    q, k, v, do = (d0[n].clone() for n in ("q", "k", "v", "do"))
    o, lse = api.attnfuse_fwd_blocksparse(q, k, v, bm, **kw)   # eager warm-up: builds the table
    api.attnfuse_bwd_blocksparse(q, k, v, o, do, lse, bm, **kw)
    o_s, lse_s = torch.empty_like(q), torch.empty(B, H, S, device="cuda")
    dq_s, dk_s, dv_s = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(api.attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, "neox"), device="cuda", dtype=torch.uint8)

    def step():
        api.attnfuse_fwd_blocksparse(q, k, v, bm, out=o_s, lse=lse_s, **kw)
        api.attnfuse_bwd_blocksparse(q, k, v, o_s, do, lse_s, bm, dq=dq_s, dk=dk_s, dv=dv_s, workspace=ws, **kw)

    g = _capture(step)
    for seed in SEEDS:
        _, d = device_inputs(B, H, Hkv, S, D, seed=seed, with_do=True)
        o_e, lse_e = api.attnfuse_fwd_blocksparse(d["q"], d["k"], d["v"], bm, **kw)
        grads_e = api.attnfuse_bwd_blocksparse(d["q"], d["k"], d["v"], o_e, d["do"], lse_e, bm, **kw)
        torch.cuda.synchronize()
        for dst, name in ((q, "q"), (k, "k"), (v, "v"), (do, "do")):
            dst.copy_(d[name])
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_s, o_e) and torch.equal(lse_s, lse_e), f"seed {seed}: forward replay differs"
        for name, a, b in zip(("dQ", "dK", "dV"), (dq_s, dk_s, dv_s), grads_e):
            assert torch.equal(a, b), f"seed {seed}: {name} replay differs"


def test_graph_decode_replays():
    """Decode (split + combine) over a ragged batch of caches with RoPE on the query."""
    need_gpu()
    announce("graph capture: decode")
    B, H, Hkv, S, D = 2, 32, 8, 3000, 128
    kw = dict(rope="neox", theta=500000.0)
    c0 = inputs.make_decode(B, H, Hkv, S, D, seed=70)
    q, kc, vc = (c0[n].cuda() for n in ("q", "k", "v"))
    lens = torch.tensor([3000, 1234], dtype=torch.int32, device="cuda")
    api.attnfuse_decode(q, kc, vc, lens, **kw)
    o_s, lse_s = torch.empty_like(q), torch.empty(B, H, device="cuda")
    ws = torch.empty(api.attnfuse_decode_workspace_bytes(B, H, Hkv, S, D), device="cuda", dtype=torch.uint8)
    g = _capture(lambda: api.attnfuse_decode(q, kc, vc, lens, out=o_s, lse=lse_s, workspace=ws, **kw))
    for seed in SEEDS:
        c = inputs.make_decode(B, H, Hkv, S, D, seed=seed)
        dq, dk, dv = (c[n].cuda() for n in ("q", "k", "v"))
        o_e, lse_e = api.attnfuse_decode(dq, dk, dv, lens, **kw)
        torch.cuda.synchronize()
        q.copy_(dq)
        kc.copy_(dk)
        vc.copy_(dv)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_s, o_e) and torch.equal(lse_s, lse_e), f"seed {seed}: replay differs"


def test_graph_separate_path_replays():
    """The separate path: Q and K rotated by the rotation kernel into buffers of
    their own, then the forward without RoPE on the rotated tensors."""
    need_gpu()
    announce("graph capture: rotation + forward without RoPE")
    B, H, Hkv, S, D = 2, 8, 2, 777, 64
    kw = dict(rope="interleaved", theta=10000.0)
    _, d0 = device_inputs(B, H, Hkv, S, D, seed=74)
    q, k, v = (d0[n].clone() for n in ("q", "k", "v"))
    api.attnfuse_rope(q, k, **kw)                       # eager warm-up: builds the table
    qr, kr = torch.empty_like(q), torch.empty_like(k)
    o_s, lse_s = torch.empty_like(q), torch.empty(B, H, S, device="cuda")

    def step():
        api.attnfuse_rope(q, k, out_q=qr, out_k=kr, **kw)
        api.attnfuse_fwd(qr, kr, v, out=o_s, lse=lse_s, mask="causal")

    g = _capture(step)
    for seed in SEEDS:
        _, d = device_inputs(B, H, Hkv, S, D, seed=seed)
        rq, rk = api.attnfuse_rope(d["q"], d["k"], **kw)
        o_e, lse_e = api.attnfuse_fwd(rq, rk, d["v"], mask="causal")
        torch.cuda.synchronize()
        for dst, name in ((q, "q"), (k, "k"), (v, "v")):
            dst.copy_(d[name])
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(qr, rq) and torch.equal(kr, rk), f"seed {seed}: rotation replay differs"
        assert torch.equal(o_s, o_e) and torch.equal(lse_s, lse_e), f"seed {seed}: forward replay differs"


@pytest.mark.parametrize("norm", ["softmax", "relu"])
def test_graph_bias_norm_replays(norm):
    """Dense bias (broadcast over heads) under softmax or relu attention, forward
    then backward; every replay gets fresh inputs and fresh bias values."""
    need_gpu()
    announce(f"graph capture: bias, norm={norm}")
    B, H, Hkv, S, D = 2, 4, 2, 300, 128
    relu = norm == "relu"
    kw = dict(norm=norm, rope="neox", mask="causal", scale=D ** -0.5 / (S if relu else 1))
    _, d0 = device_inputs(B, H, Hkv, S, D, seed=75, with_do=True)
    q, k, v, do = (d0[n].clone() for n in ("q", "k", "v", "do"))
    bias = torch.zeros(B, 1, S, S, device="cuda")
    o, lse = api.attnfuse_fwd_bias_norm(q, k, v, bias=bias, **kw)   # eager warm-up: builds the table
    api.attnfuse_bwd_bias_norm(q, k, v, o, do, lse, bias=bias, **kw)
    o_s = torch.empty_like(q)
    lse_s = None if relu else torch.empty(B, H, S, device="cuda")
    dq_s, dk_s, dv_s = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(api.attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, "neox"), device="cuda", dtype=torch.uint8)

    def step():
        api.attnfuse_fwd_bias_norm(q, k, v, bias=bias, out=o_s, lse=lse_s, **kw)
        api.attnfuse_bwd_bias_norm(q, k, v, o_s, do, lse_s, bias=bias, dq=dq_s, dk=dk_s, dv=dv_s, workspace=ws, **kw)

    g = _capture(step)
    for seed in SEEDS:
        _, d = device_inputs(B, H, Hkv, S, D, seed=seed, with_do=True)
        gen = torch.Generator("cpu").manual_seed(seed)
        b_new = (torch.randn(B, 1, S, S, generator=gen) / (S if relu else 1)).cuda()
        o_e, lse_e = api.attnfuse_fwd_bias_norm(d["q"], d["k"], d["v"], bias=b_new, **kw)
        grads_e = api.attnfuse_bwd_bias_norm(d["q"], d["k"], d["v"], o_e, d["do"], lse_e, bias=b_new, **kw)
        torch.cuda.synchronize()
        for dst, name in ((q, "q"), (k, "k"), (v, "v"), (do, "do")):
            dst.copy_(d[name])
        bias.copy_(b_new)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o_s, o_e), f"seed {seed}: forward replay differs"
        if not relu:
            assert torch.equal(lse_s, lse_e), f"seed {seed}: LSE replay differs"
        for name, a, b in zip(("dQ", "dK", "dV"), (dq_s, dk_s, dv_s), grads_e):
            assert torch.equal(a, b), f"seed {seed}: {name} replay differs"
