"""Python binding of the C ABI in include/attnfuse.h -- argument marshalling only.

Each function takes torch tensors that already live on the GPU, checks their
shape/dtype/contiguity against the call, passes raw device pointers and the
current torch stream to the library, and raises AttnFuseError on a non-zero
return code.  Every step of the computation runs in the HIP kernels.
"""
import math

import torch

from . import _lib

DTYPE = {torch.bfloat16: 0, torch.float32: 1}
ROPE = {"none": 0, "neox": 1, "interleaved": 2}
MASK = {"none": 0, "causal": 1, "sliding_window": 2}


class AttnFuseError(RuntimeError):
    def __init__(self, code, where):
        msg = _lib.load().attnfuse_strerror(code).decode()
        super().__init__(f"{where}: {msg} (code {code})")
        self.code = code


def _check(code, where):
    if code != 0:
        raise AttnFuseError(code, where)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def _shape(q, k):
    if q.dim() != 4 or k.dim() != 4:
        raise ValueError("q must be [B, H, S, D] and k/v [B, H_kv, S, D]")
    B, H, S, D = q.shape
    if k.shape[0] != B or k.shape[2] != S or k.shape[3] != D:
        raise ValueError("k/v must be [B, H_kv, S, D] matching q")
    return B, H, k.shape[1], S, D


def _same(ref, *ts):
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda or t.dtype != ref.dtype or not t.is_contiguous():
            raise ValueError("tensors must be contiguous, on the GPU, and share one dtype")


def _variant(rope, theta, mask, window, alibi_slopes, scale, D):
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if alibi_slopes is not None and (alibi_slopes.dtype != torch.float32 or not alibi_slopes.is_cuda):
        raise ValueError("alibi_slopes must be an fp32 GPU tensor [H]")
    return ROPE[rope], float(theta), MASK[mask], int(window or 0), scale


def attnfuse_fwd(q, k, v, *, rope="none", theta=10000.0, mask="causal", window=None,
                 alibi_slopes=None, scale=None, out=None, lse=None):
    """O, LSE = attention(q, k, v); see attnfuse_fwd in include/attnfuse.h."""
    B, H, Hkv, S, D = _shape(q, k)
    _same(q, k, v, out)
    if v.shape != k.shape:
        raise ValueError("v must have k's shape")
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(B, H, S, device=q.device, dtype=torch.float32) if lse is None else lse
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D)
    code = _lib.load().attnfuse_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, H, Hkv, S, D,
                                    DTYPE[q.dtype], r, th, m, w, _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_fwd")
    return out, lse


def attnfuse_bwd_workspace_bytes(B, H, H_kv, S, D, rope="none"):
    return _lib.load().attnfuse_bwd_workspace_bytes(B, H, H_kv, S, D, ROPE[rope])


def attnfuse_bwd(q, k, v, o, do, lse, *, rope="none", theta=10000.0, mask="causal", window=None,
                 alibi_slopes=None, scale=None, dq=None, dk=None, dv=None, workspace=None):
    """dQ, dK, dV of attnfuse_fwd; see attnfuse_bwd in include/attnfuse.h."""
    B, H, Hkv, S, D = _shape(q, k)
    _same(q, k, v, o, do, dq, dk, dv)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    nbytes = attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, rope)
    if workspace is None:
        workspace = torch.empty(nbytes, device=q.device, dtype=torch.uint8)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D)
    code = _lib.load().attnfuse_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                    _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), workspace.numel(),
                                    B, H, Hkv, S, D, DTYPE[q.dtype], r, th, m, w,
                                    _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_bwd")
    return dq, dk, dv


def _mask_ptrs(block_mask, q, S):
    if block_mask.S != S:
        raise ValueError(f"block mask built for S={block_mask.S}, tensors have S={S}")
    ts = (block_mask.q_ptr, block_mask.k_idx, block_mask.k_ptr, block_mask.q_idx)
    for t in ts:
        if t.device != q.device or t.dtype != torch.int32 or not t.is_contiguous():
            raise ValueError("block mask lists must be contiguous int32 tensors on q's device")
    # an empty index list has no storage; any valid aligned address serves
    return [t.data_ptr() if t.numel() else block_mask.q_ptr.data_ptr() for t in ts]


def attnfuse_fwd_blocksparse(q, k, v, block_mask, *, rope="none", theta=10000.0, mask="none", window=None,
                             alibi_slopes=None, scale=None, out=None, lse=None):
    """O, LSE of attention restricted to the active blocks of ``block_mask``
    (a blockmask.BlockMask); see attnfuse_fwd_blocksparse."""
    B, H, Hkv, S, D = _shape(q, k)
    _same(q, k, v, out)
    if v.shape != k.shape:
        raise ValueError("v must have k's shape")
    qp, ki, _, _ = _mask_ptrs(block_mask, q, S)
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(B, H, S, device=q.device, dtype=torch.float32) if lse is None else lse
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D)
    code = _lib.load().attnfuse_fwd_blocksparse(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), qp, ki,
                                                B, H, Hkv, S, D, DTYPE[q.dtype], r, th, m, w, _ptr(alibi_slopes),
                                                sc, _stream())
    _check(code, "attnfuse_fwd_blocksparse")
    return out, lse


def attnfuse_bwd_blocksparse(q, k, v, o, do, lse, block_mask, *, rope="none", theta=10000.0, mask="none",
                             window=None, alibi_slopes=None, scale=None, dq=None, dk=None, dv=None,
                             workspace=None):
    """dQ, dK, dV of attnfuse_fwd_blocksparse; see attnfuse_bwd_blocksparse."""
    B, H, Hkv, S, D = _shape(q, k)
    _same(q, k, v, o, do, dq, dk, dv)
    qp, ki, kp, qi = _mask_ptrs(block_mask, q, S)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    nbytes = attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, rope)
    if workspace is None:
        workspace = torch.empty(nbytes, device=q.device, dtype=torch.uint8)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D)
    code = _lib.load().attnfuse_bwd_blocksparse(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                                _ptr(dq), _ptr(dk), _ptr(dv), qp, ki, kp, qi, _ptr(workspace),
                                                workspace.numel(), B, H, Hkv, S, D, DTYPE[q.dtype], r, th, m, w,
                                                _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_bwd_blocksparse")
    return dq, dk, dv


NORM = {"softmax": 0, "relu": 1}


def _bias_args(bias, q, B, H, S):
    """(pointer, stride_b, stride_h, stride_q) of an fp32 GPU bias broadcastable
    to [B, H, S, S] with keys contiguous (broadcast dimensions get stride 0)."""
    if bias is None:
        return None, 0, 0, 0
    if bias.dtype != torch.float32 or bias.device != q.device:
        raise ValueError("bias must be an fp32 tensor on q's device")
    while bias.dim() < 4:
        bias = bias.unsqueeze(0)
    e = bias.expand(B, H, S, S)
    if e.stride(3) != 1:
        raise ValueError("bias must be contiguous along the key dimension")
    return e.data_ptr(), e.stride(0), e.stride(1), e.stride(2)


def attnfuse_fwd_bias_norm(q, k, v, *, bias=None, norm="softmax", rope="none", theta=10000.0, mask="causal",
                           window=None, scale=None, out=None, lse=None):
    """O (and LSE, None under relu attention) with a dense additive bias and/or
    relu attention; see attnfuse_fwd_bias_norm in include/attnfuse.h."""
    B, H, Hkv, S, D = _shape(q, k)
    _same(q, k, v, out)
    if v.shape != k.shape:
        raise ValueError("v must have k's shape")
    out = torch.empty_like(q) if out is None else out
    if NORM[norm] == NORM["softmax"] and lse is None:
        lse = torch.empty(B, H, S, device=q.device, dtype=torch.float32)
    bp, sb, sh, sq = _bias_args(bias, q, B, H, S)
    r, th, m, w, sc = _variant(rope, theta, mask, window, None, scale, D)
    code = _lib.load().attnfuse_fwd_bias_norm(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), bp, sb, sh, sq,
                                              NORM[norm], B, H, Hkv, S, D, DTYPE[q.dtype], r, th, m, w, None, sc,
                                              _stream())
    _check(code, "attnfuse_fwd_bias_norm")
    return out, lse


def attnfuse_bwd_bias_norm(q, k, v, o, do, lse, *, bias=None, norm="softmax", rope="none", theta=10000.0,
                           mask="causal", window=None, scale=None, dq=None, dk=None, dv=None, workspace=None):
    """dQ, dK, dV of attnfuse_fwd_bias_norm (lse may be None under relu
    attention); see attnfuse_bwd_bias_norm."""
    B, H, Hkv, S, D = _shape(q, k)
    _same(q, k, v, o, do, dq, dk, dv)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    nbytes = attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, rope)
    if workspace is None:
        workspace = torch.empty(nbytes, device=q.device, dtype=torch.uint8)
    bp, sb, sh, sq = _bias_args(bias, q, B, H, S)
    r, th, m, w, sc = _variant(rope, theta, mask, window, None, scale, D)
    code = _lib.load().attnfuse_bwd_bias_norm(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                              _ptr(dq), _ptr(dk), _ptr(dv), bp, sb, sh, sq, NORM[norm],
                                              _ptr(workspace), workspace.numel(), B, H, Hkv, S, D, DTYPE[q.dtype],
                                              r, th, m, w, None, sc, _stream())
    _check(code, "attnfuse_bwd_bias_norm")
    return dq, dk, dv


def attnfuse_decode_workspace_bytes(B, H, H_kv, S_kv, D):
    return _lib.load().attnfuse_decode_workspace_bytes(B, H, H_kv, S_kv, D)


def attnfuse_decode(q, k_cache, v_cache, cache_lens=None, *, rope="none", theta=10000.0, mask="causal",
                    window=None, alibi_slopes=None, scale=None, out=None, lse=None, workspace=None):
    """O [B,H,D], LSE [B,H] of one query per sequence against a KV cache of
    already-rotated keys; see attnfuse_decode in include/attnfuse.h."""
    if q.dim() != 3 or k_cache.dim() != 4 or v_cache.shape != k_cache.shape:
        raise ValueError("q must be [B, H, D] and the caches [B, H_kv, S_kv, D]")
    B, H, D = q.shape
    Hkv, S_kv = k_cache.shape[1], k_cache.shape[2]
    if k_cache.shape[0] != B or k_cache.shape[3] != D:
        raise ValueError("cache shape does not match q")
    _same(q, k_cache, v_cache, out)
    if cache_lens is not None and (cache_lens.dtype != torch.int32 or not cache_lens.is_cuda
                                   or cache_lens.shape != (B,)):
        raise ValueError("cache_lens must be an int32 GPU tensor [B]")
    out = torch.empty_like(q) if out is None else out
    lse = torch.empty(B, H, device=q.device, dtype=torch.float32) if lse is None else lse
    nbytes = attnfuse_decode_workspace_bytes(B, H, Hkv, S_kv, D)
    if workspace is None:
        workspace = torch.empty(nbytes, device=q.device, dtype=torch.uint8)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D)
    code = _lib.load().attnfuse_decode(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(cache_lens), _ptr(out),
                                       _ptr(lse), _ptr(workspace), workspace.numel(), B, H, Hkv, S_kv, D,
                                       DTYPE[q.dtype], r, th, m, w, _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_decode")
    return out, lse


def _rope_call(name, x0, x1, y0, y1, rope, theta):
    if x1 is not None:
        B, H, Hkv, S, D = _shape(x0, x1)
    else:
        B, H, S, D = x0.shape
        Hkv = 1
    _same(x0, x1, y0, y1)
    y0 = torch.empty_like(x0) if y0 is None else y0
    if x1 is not None and y1 is None:
        y1 = torch.empty_like(x1)
    code = getattr(_lib.load(), name)(_ptr(x0), _ptr(x1), _ptr(y0), _ptr(y1), B, H, Hkv, S, D,
                                      DTYPE[x0.dtype], ROPE[rope], float(theta), _stream())
    _check(code, name)
    return y0, y1


def attnfuse_rope(q, k=None, *, rope="neox", theta=10000.0, out_q=None, out_k=None):
    """Qr, Kr = R q, R k (separate pre-rotation); see attnfuse_rope."""
    return _rope_call("attnfuse_rope", q, k, out_q, out_k, rope, theta)


def attnfuse_rope_bwd(dqr, dkr=None, *, rope="neox", theta=10000.0, out_q=None, out_k=None):
    """dQ, dK = R^T dQr, R^T dKr; see attnfuse_rope_bwd."""
    return _rope_call("attnfuse_rope_bwd", dqr, dkr, out_q, out_k, rope, theta)


def attnfuse_strerror(code):
    return _lib.load().attnfuse_strerror(code).decode()


def attnfuse_version():
    return _lib.load().attnfuse_version()
