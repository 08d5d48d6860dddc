"""The Python binding's argument checks (CPU): every tensor, q included, must
be contiguous, of the call's dtype and exact shape, and on q's device before
any pointer reaches the library; a caller's workspace counts its bytes, not
its elements."""
import pytest
import torch

from paper_2609_13612_amd import api

CPU = torch.device("cpu")


def test_need_accepts_exact_tensor():
    api._need(torch.zeros(2, 3, 4, dtype=torch.bfloat16), "x", (2, 3, 4), torch.bfloat16, CPU)


@pytest.mark.parametrize("bad,why", [
    (torch.zeros(2, 3, 5, dtype=torch.bfloat16), "shape"),
    (torch.zeros(2, 3, 4, dtype=torch.float32), "must be torch.bfloat16"),
    (torch.zeros(2, 4, 3, dtype=torch.bfloat16).transpose(1, 2), "contiguous"),
    (torch.zeros(2, 3, 4, dtype=torch.bfloat16, device="meta"), "on cpu"),
])
def test_need_rejects(bad, why):
    with pytest.raises(ValueError, match=why):
        api._need(bad, "x", (2, 3, 4), torch.bfloat16, CPU)


def test_need_rejects_non_tensor():
    with pytest.raises(TypeError):
        api._need([1, 2], "x", (2,), torch.float32, CPU)


def test_opt_allocates_or_checks():
    t = api._opt(None, "out", (2, 3), torch.float32, CPU)
    assert t.shape == (2, 3) and t.dtype == torch.float32
    with pytest.raises(ValueError, match="shape"):
        api._opt(torch.zeros(2, 2), "out", (2, 3), torch.float32, CPU)


def test_workspace_counts_bytes():
    ws, n = api._workspace(None, 1000, CPU)
    assert ws.dtype == torch.uint8 and n == 1000
    ws, n = api._workspace(torch.zeros(300, dtype=torch.float32), 1000, CPU)
    assert n == 1200                      # 300 fp32 elements are 1200 bytes
    with pytest.raises(ValueError):
        api._workspace(torch.zeros(300, 2).t(), 1000, CPU)


def test_backward_inputs_checked():
    q = torch.zeros(1, 4, 8, 64, dtype=torch.bfloat16)
    k = torch.zeros(1, 2, 8, 64, dtype=torch.bfloat16)
    lse = torch.zeros(1, 4, 8)
    api._bwd_inputs(q, k, k, q, q, lse, CPU, lse_needed=True)
    with pytest.raises(ValueError, match="do"):
        api._bwd_inputs(q, k, k, q, q[:, :2], lse, CPU, lse_needed=True)
    with pytest.raises(ValueError, match="lse"):
        api._bwd_inputs(q, k, k, q, q, lse[:, :, :4], CPU, lse_needed=True)
    with pytest.raises(TypeError):
        api._bwd_inputs(q, k, k, q, q, None, CPU, lse_needed=True)
    api._bwd_inputs(q, k, k, q, q, None, CPU, lse_needed=False)   # relu attention: no LSE


def test_cpu_q_is_rejected_before_the_library():
    q = torch.zeros(1, 2, 8, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU"):
        api.attnfuse_fwd(q, q, q)
    with pytest.raises(ValueError, match="GPU"):
        api.attnfuse_decode(q[:, :, 0], q, q)
    with pytest.raises(ValueError, match="GPU"):
        api.attnfuse_rope(q)


def test_block_mask_offset_lengths_checked():
    from paper_2609_13612_amd import blockmask
    bm = blockmask.block_mask_from_dense(torch.ones(3, 3, dtype=torch.bool), 150)
    q = torch.zeros(1, 1, 150, 64, dtype=torch.bfloat16)
    assert len(api._mask_ptrs(bm, q, 150)) == 4
    short = blockmask.BlockMask(bm.S, bm.active, bm.q_ptr[:-1].contiguous(), bm.k_idx, bm.k_ptr, bm.q_idx)
    with pytest.raises(ValueError, match="nb \\+ 1"):
        api._mask_ptrs(short, q, 150)


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    """No fallback: without the built library every entry point raises."""
    from paper_2609_13612_amd import _lib
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "libattnfuse.so"))
    monkeypatch.setattr(_lib, "_lib", None)
    with pytest.raises(FileNotFoundError, match="no non-HIP fallback"):
        _lib.load()
    with pytest.raises(FileNotFoundError):
        api.attnfuse_bwd_workspace_bytes(1, 1, 1, 64, 64)


def test_package_never_uses_the_oracle():
    """The oracle is test infrastructure: no module of the package imports it,
    and none falls back to a torch attention routine."""
    import pathlib
    import re
    pkg = pathlib.Path(api.__file__).parent
    for f in sorted(pkg.rglob("*.py")):
        text = f.read_text()
        assert not re.search(r"^\s*(import|from)\s+oracle\b", text, flags=re.M), f"{f.name} imports the oracle"
        assert "scaled_dot_product_attention" not in text, f"{f.name} calls a torch attention routine"
