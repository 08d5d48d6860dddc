"""The library keeps no per-call state: two different problems issued at the
same time on two streams (default priority) each give exactly their own
results from a single stream (GPU)."""
import pytest
import torch

from gpu_util import announce, device_inputs, need_gpu
from paper_2609_13612_amd import api

pytestmark = pytest.mark.gpu

PROBLEMS = {
    "a": ((1, 8, 2, 700, 128), dict(rope="neox", theta=500000.0, mask="causal")),
    "b": ((2, 4, 4, 513, 64), dict(rope="interleaved", theta=10000.0, mask="sliding_window", window=100)),
}


def _run(d, shape, kw, out):
    B, H, Hkv, S, D = shape
    api.attnfuse_fwd(d["q"], d["k"], d["v"], out=out["o"], lse=out["lse"], **kw)
    api.attnfuse_bwd(d["q"], d["k"], d["v"], out["o"], d["do"], out["lse"], dq=out["dq"], dk=out["dk"], dv=out["dv"],
                     workspace=out["ws"], **kw)


def _outputs(shape, kw):
    B, H, Hkv, S, D = shape
    return {"o": torch.empty(B, H, S, D, device="cuda", dtype=torch.bfloat16),
            "lse": torch.empty(B, H, S, device="cuda"),
            "dq": torch.empty(B, H, S, D, device="cuda", dtype=torch.bfloat16),
            "dk": torch.empty(B, Hkv, S, D, device="cuda", dtype=torch.bfloat16),
            "dv": torch.empty(B, Hkv, S, D, device="cuda", dtype=torch.bfloat16),
            "ws": torch.empty(api.attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, kw["rope"]), device="cuda",
                              dtype=torch.uint8)}


def test_two_streams_at_once_match_single_stream():
    need_gpu()
    announce("two streams at once")
    ins, refs, outs = {}, {}, {}
    for i, (name, (shape, kw)) in enumerate(PROBLEMS.items()):
        _, ins[name] = device_inputs(*shape, seed=80 + i, with_do=True)
        refs[name] = _outputs(shape, kw)
        _run(ins[name], shape, kw, refs[name])                    # single stream, one after the other
        outs[name] = _outputs(shape, kw)
    torch.cuda.synchronize()
    streams = {name: torch.cuda.Stream() for name in PROBLEMS}
    for _ in range(3):                                            # interleaved launches on both streams
        for name, (shape, kw) in PROBLEMS.items():
            with torch.cuda.stream(streams[name]):
                _run(ins[name], shape, kw, outs[name])
    torch.cuda.synchronize()
    for name in PROBLEMS:
        for key in ("o", "lse", "dq", "dk", "dv"):
            assert torch.equal(outs[name][key], refs[name][key]), f"problem {name}: {key} differs on its own stream"
