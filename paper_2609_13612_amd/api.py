"""Python binding of the C ABI in include/attnfuse.h -- argument marshalling only.

Each function takes torch tensors that already live on the GPU, checks their
shape/dtype/contiguity against the call, passes raw device pointers and the
current torch stream to the library, and raises AttnFuseError on a non-zero
return code.  Every step of the computation runs in the HIP kernels.
"""
import math

import numpy as np
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


def _device(q):
    """The GPU that q lives on (every other tensor of the call must be there too)."""
    if not isinstance(q, torch.Tensor) or not q.is_cuda:
        raise ValueError("q must be a tensor on a GPU")
    if q.dtype not in DTYPE:
        raise ValueError(f"dtype must be one of {sorted(str(d) for d in DTYPE)}")
    return q.device


def _need(t, name, shape, dtype, device):
    """Raise unless t is a contiguous tensor of exactly that shape and dtype on device."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device != device:
        raise ValueError(f"{name} must be on {device} (it is on {t.device})")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (it is {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (it has {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _opt(t, name, shape, dtype, device):
    """A caller-provided output: checked like an input, or allocated."""
    if t is None:
        return torch.empty(shape, device=device, dtype=dtype)
    _need(t, name, shape, dtype, device)
    return t


def _inputs(q, k, v, device):
    """q [B, H, S, D]; k and v [B, H_kv, S, D] of q's dtype, all on q's device."""
    _need(q, "q", q.shape, q.dtype, device)
    _need(k, "k", k.shape, q.dtype, device)
    _need(v, "v", k.shape, q.dtype, device)


def _bwd_inputs(q, k, v, o, do, lse, device, lse_needed):
    _inputs(q, k, v, device)
    _need(o, "o", q.shape, q.dtype, device)
    _need(do, "do", q.shape, q.dtype, device)
    if lse is not None or lse_needed:
        _need(lse, "lse", q.shape[:3], torch.float32, device)


def _grads(q, k, dq, dk, dv, device):
    return (_opt(dq, "dq", q.shape, q.dtype, device), _opt(dk, "dk", k.shape, q.dtype, device),
            _opt(dv, "dv", k.shape, q.dtype, device))


def _workspace(ws, nbytes, device):
    """(tensor, size in bytes) of the workspace: the caller's, checked, or a new one."""
    if ws is None:
        return torch.empty(nbytes, device=device, dtype=torch.uint8), nbytes
    if not isinstance(ws, torch.Tensor) or ws.device != device or not ws.is_contiguous():
        raise ValueError("workspace must be a contiguous tensor on q's device")
    return ws, ws.numel() * ws.element_size()


# RoPE cos/sin tables this binding built, per (device index, D, theta): a list
# of tables (each a [rows, D/2, 2] fp32 tensor), never freed, since a kernel
# on any stream may still read one.  The library itself keeps nothing.
_TABLES = {}
_TABLE_MIN_ROWS = 4096


def rope_table(D, theta, rows, device=None, out=None):
    """A RoPE cos/sin table for positions 0..rows-1: T[n][i] = (cos, sin) of
    n * theta^(-2i/D), filled by attnfuse_rope_table_fill on the current stream
    (see include/attnfuse.h).  Pass it as ``rope_table=`` to any call with the
    same D and theta and S <= rows."""
    device = torch.device("cuda", torch.cuda.current_device()) if device is None else torch.device(device)
    shape = (rows, D // 2, 2)
    if out is None:
        out = torch.empty(shape, device=device, dtype=torch.float32)
    else:
        _need(out, "out", shape, torch.float32, device)
    with torch.cuda.device(device):
        code = _lib.load().attnfuse_rope_table_fill(out.data_ptr(), rows, D, float(theta), _stream())
    _check(code, "attnfuse_rope_table_fill")
    return out


def _table(rope, theta, D, S, device, given):
    """The cos/sin table a call reads, as a tensor: the caller's (checked), or
    one this binding keeps for (device, D, theta).  Under HIP graph capture a
    table not yet built is filled inside the capture (stream-ordered before the
    call that reads it) and not kept; the caller holds the returned tensor
    until its launch is enqueued.  None without RoPE."""
    if ROPE[rope] == ROPE["none"]:
        return None
    if given is not None:
        if (not isinstance(given, torch.Tensor) or given.device != device or given.dtype != torch.float32
                or given.dim() != 3 or tuple(given.shape[1:]) != (D // 2, 2) or not given.is_contiguous()):
            raise ValueError(f"rope_table must be a contiguous fp32 [rows, {D // 2}, 2] tensor on {device}")
        if given.shape[0] < S:
            raise ValueError(f"rope_table has {given.shape[0]} rows, the call needs {S}")
        return given
    key = (device.index, D, float(np.float32(theta)))
    for t in _TABLES.get(key, ()):
        if t.shape[0] >= S:
            return t
    rows = _TABLE_MIN_ROWS
    while rows < S:
        rows *= 2
    with torch.cuda.device(device):
        if torch.cuda.is_current_stream_capturing():
            return rope_table(D, theta, S, device)
        t = rope_table(D, theta, rows, device)
        # ready for any stream before it is shared: one wait, once per table
        torch.cuda.current_stream().synchronize()
    _TABLES.setdefault(key, []).append(t)
    return t


def _tab(t):
    """(pointer, rows) of a table from _table."""
    return (None, 0) if t is None else (t.data_ptr(), t.shape[0])


def _variant(rope, theta, mask, window, alibi_slopes, scale, D, H=None, device=None):
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if alibi_slopes is not None:
        _need(alibi_slopes, "alibi_slopes", (H,), torch.float32, device)
    return ROPE[rope], float(theta), MASK[mask], int(window or 0), scale


def attnfuse_fwd(q, k, v, *, rope="none", theta=10000.0, mask="causal", window=None,
                 alibi_slopes=None, scale=None, out=None, lse=None, rope_table=None):
    """O, LSE = attention(q, k, v); see attnfuse_fwd in include/attnfuse.h."""
    dev = _device(q)
    B, H, Hkv, S, D = _shape(q, k)
    _inputs(q, k, v, dev)
    out = _opt(out, "out", q.shape, q.dtype, dev)
    lse = _opt(lse, "lse", (B, H, S), torch.float32, dev)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D, H, dev)
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, H, Hkv, S, D,
                                        DTYPE[q.dtype], r, th, tp, tr, m, w, _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_fwd")
    return out, lse


def attnfuse_bwd_workspace_bytes(B, H, H_kv, S, D, rope="none"):
    return _lib.load().attnfuse_bwd_workspace_bytes(B, H, H_kv, S, D, ROPE[rope])


def attnfuse_bwd(q, k, v, o, do, lse, *, rope="none", theta=10000.0, mask="causal", window=None,
                 alibi_slopes=None, scale=None, dq=None, dk=None, dv=None, workspace=None, rope_table=None):
    """dQ, dK, dV of attnfuse_fwd; see attnfuse_bwd in include/attnfuse.h."""
    dev = _device(q)
    B, H, Hkv, S, D = _shape(q, k)
    _bwd_inputs(q, k, v, o, do, lse, dev, lse_needed=True)
    dq, dk, dv = _grads(q, k, dq, dk, dv, dev)
    workspace, wbytes = _workspace(workspace, attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, rope), dev)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D, H, dev)
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_bwd(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                        _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), wbytes,
                                        B, H, Hkv, S, D, DTYPE[q.dtype], r, th, tp, tr, m, w,
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
    # the offset arrays are read up to entry nb; their values are those the
    # blockmask constructors built and checked
    nb = (S + 63) // 64
    if block_mask.q_ptr.numel() != nb + 1 or block_mask.k_ptr.numel() != nb + 1:
        raise ValueError(f"block mask offset lists must have nb + 1 = {nb + 1} entries")
    # an empty index list has no storage; any valid aligned address serves
    return [t.data_ptr() if t.numel() else block_mask.q_ptr.data_ptr() for t in ts]


def attnfuse_fwd_blocksparse(q, k, v, block_mask, *, rope="none", theta=10000.0, mask="none", window=None,
                             alibi_slopes=None, scale=None, out=None, lse=None, rope_table=None):
    """O, LSE of attention restricted to the active blocks of ``block_mask``
    (a blockmask.BlockMask); see attnfuse_fwd_blocksparse."""
    dev = _device(q)
    B, H, Hkv, S, D = _shape(q, k)
    _inputs(q, k, v, dev)
    qp, ki, _, _ = _mask_ptrs(block_mask, q, S)
    out = _opt(out, "out", q.shape, q.dtype, dev)
    lse = _opt(lse, "lse", (B, H, S), torch.float32, dev)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D, H, dev)
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_fwd_blocksparse(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), qp, ki,
                                                    B, H, Hkv, S, D, DTYPE[q.dtype], r, th, tp, tr, m, w,
                                                    _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_fwd_blocksparse")
    return out, lse


def attnfuse_bwd_blocksparse(q, k, v, o, do, lse, block_mask, *, rope="none", theta=10000.0, mask="none",
                             window=None, alibi_slopes=None, scale=None, dq=None, dk=None, dv=None,
                             workspace=None, rope_table=None):
    """dQ, dK, dV of attnfuse_fwd_blocksparse; see attnfuse_bwd_blocksparse."""
    dev = _device(q)
    B, H, Hkv, S, D = _shape(q, k)
    _bwd_inputs(q, k, v, o, do, lse, dev, lse_needed=True)
    qp, ki, kp, qi = _mask_ptrs(block_mask, q, S)
    dq, dk, dv = _grads(q, k, dq, dk, dv, dev)
    workspace, wbytes = _workspace(workspace, attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, rope), dev)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D, H, dev)
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_bwd_blocksparse(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                                    _ptr(dq), _ptr(dk), _ptr(dv), qp, ki, kp, qi, _ptr(workspace),
                                                    wbytes, B, H, Hkv, S, D, DTYPE[q.dtype], r, th, tp, tr, m, w,
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
                           window=None, scale=None, out=None, lse=None, rope_table=None):
    """O (and LSE, None under relu attention) with a dense additive bias and/or
    relu attention; see attnfuse_fwd_bias_norm in include/attnfuse.h."""
    dev = _device(q)
    B, H, Hkv, S, D = _shape(q, k)
    _inputs(q, k, v, dev)
    out = _opt(out, "out", q.shape, q.dtype, dev)
    if NORM[norm] == NORM["softmax"] or lse is not None:
        lse = _opt(lse, "lse", (B, H, S), torch.float32, dev)
    bp, sb, sh, sq = _bias_args(bias, q, B, H, S)
    r, th, m, w, sc = _variant(rope, theta, mask, window, None, scale, D)
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_fwd_bias_norm(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), bp, sb, sh,
                                                  sq, NORM[norm], B, H, Hkv, S, D, DTYPE[q.dtype], r, th, tp, tr, m, w,
                                                  None, sc, _stream())
    _check(code, "attnfuse_fwd_bias_norm")
    return out, lse


def attnfuse_bwd_bias_norm(q, k, v, o, do, lse, *, bias=None, norm="softmax", rope="none", theta=10000.0,
                           mask="causal", window=None, scale=None, dq=None, dk=None, dv=None, workspace=None,
                           rope_table=None):
    """dQ, dK, dV of attnfuse_fwd_bias_norm (lse may be None under relu
    attention); see attnfuse_bwd_bias_norm."""
    dev = _device(q)
    B, H, Hkv, S, D = _shape(q, k)
    _bwd_inputs(q, k, v, o, do, lse, dev, lse_needed=NORM[norm] == NORM["softmax"])
    dq, dk, dv = _grads(q, k, dq, dk, dv, dev)
    workspace, wbytes = _workspace(workspace, attnfuse_bwd_workspace_bytes(B, H, Hkv, S, D, rope), dev)
    bp, sb, sh, sq = _bias_args(bias, q, B, H, S)
    r, th, m, w, sc = _variant(rope, theta, mask, window, None, scale, D)
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_bwd_bias_norm(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse),
                                                  _ptr(dq), _ptr(dk), _ptr(dv), bp, sb, sh, sq, NORM[norm],
                                                  _ptr(workspace), wbytes, B, H, Hkv, S, D, DTYPE[q.dtype],
                                                  r, th, tp, tr, m, w, None, sc, _stream())
    _check(code, "attnfuse_bwd_bias_norm")
    return dq, dk, dv


def attnfuse_decode_workspace_bytes(B, H, H_kv, S_kv, D):
    return _lib.load().attnfuse_decode_workspace_bytes(B, H, H_kv, S_kv, D)


def _decode_args(q, k_cache, v_cache, cache_lens, out, lse):
    dev = _device(q)
    if q.dim() != 3 or k_cache.dim() != 4 or v_cache.shape != k_cache.shape:
        raise ValueError("q must be [B, H, D] and the caches [B, H_kv, S_kv, D]")
    B, H, D = q.shape
    Hkv, S_kv = k_cache.shape[1], k_cache.shape[2]
    if k_cache.shape[0] != B or k_cache.shape[3] != D:
        raise ValueError("cache shape does not match q")
    _need(q, "q", q.shape, q.dtype, dev)
    _need(k_cache, "k_cache", k_cache.shape, q.dtype, dev)
    _need(v_cache, "v_cache", k_cache.shape, q.dtype, dev)
    if cache_lens is not None:
        _need(cache_lens, "cache_lens", (B,), torch.int32, dev)
    out = _opt(out, "out", q.shape, q.dtype, dev)
    lse = _opt(lse, "lse", (B, H), torch.float32, dev)
    return dev, (B, H, Hkv, S_kv, D), out, lse


def attnfuse_decode(q, k_cache, v_cache, cache_lens=None, *, rope="none", theta=10000.0, mask="causal",
                    window=None, alibi_slopes=None, scale=None, out=None, lse=None, workspace=None,
                    rope_table=None):
    """O [B,H,D], LSE [B,H] of one query per sequence against a KV cache of
    already-rotated keys; see attnfuse_decode in include/attnfuse.h."""
    dev, (B, H, Hkv, S_kv, D), out, lse = _decode_args(q, k_cache, v_cache, cache_lens, out, lse)
    workspace, wbytes = _workspace(workspace, attnfuse_decode_workspace_bytes(B, H, Hkv, S_kv, D), dev)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D, H, dev)
    tab = _table(rope, theta, D, S_kv, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_decode(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(cache_lens), _ptr(out),
                                           _ptr(lse), _ptr(workspace), wbytes, B, H, Hkv, S_kv, D,
                                           DTYPE[q.dtype], r, th, tp, tr, m, w, _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_decode")
    return out, lse


def attnfuse_decode_noalloc(q, k_cache, v_cache, cache_lens=None, *, rope="none", theta=10000.0, mask="causal",
                            window=None, alibi_slopes=None, scale=None, out=None, lse=None, rope_table=None):
    """attnfuse_decode with the library's static scratch in place of a
    workspace; see attnfuse_decode_noalloc in include/attnfuse.h.  Pass
    ``out``, ``lse`` (and, with RoPE, ``rope_table``) for a call that
    allocates nothing at all."""
    dev, (B, H, Hkv, S_kv, D), out, lse = _decode_args(q, k_cache, v_cache, cache_lens, out, lse)
    r, th, m, w, sc = _variant(rope, theta, mask, window, alibi_slopes, scale, D, H, dev)
    tab = _table(rope, theta, D, S_kv, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = _lib.load().attnfuse_decode_noalloc(_ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(cache_lens),
                                                   _ptr(out), _ptr(lse), B, H, Hkv, S_kv, D, DTYPE[q.dtype], r, th,
                                                   tp, tr, m, w, _ptr(alibi_slopes), sc, _stream())
    _check(code, "attnfuse_decode_noalloc")
    return out, lse


def _rope_call(name, x0, x1, y0, y1, rope, theta, rope_table):
    dev = _device(x0)
    if x1 is not None:
        B, H, Hkv, S, D = _shape(x0, x1)
        _need(x1, "k", x1.shape, x0.dtype, dev)
    else:
        if x0.dim() != 4:
            raise ValueError("q must be [B, H, S, D]")
        B, H, S, D = x0.shape
        Hkv = 1
    _need(x0, "q", x0.shape, x0.dtype, dev)
    y0 = _opt(y0, "out_q", x0.shape, x0.dtype, dev)
    if x1 is not None:
        y1 = _opt(y1, "out_k", x1.shape, x0.dtype, dev)
    elif y1 is not None:
        raise ValueError("out_k needs k")
    tab = _table(rope, theta, D, S, dev, rope_table)
    tp, tr = _tab(tab)
    with torch.cuda.device(dev):
        code = getattr(_lib.load(), name)(_ptr(x0), _ptr(x1), _ptr(y0), _ptr(y1), B, H, Hkv, S, D,
                                          DTYPE[x0.dtype], ROPE[rope], float(theta), tp, tr, _stream())
    _check(code, name)
    return y0, y1


def attnfuse_rope(q, k=None, *, rope="neox", theta=10000.0, out_q=None, out_k=None, rope_table=None):
    """Qr, Kr = R q, R k (separate pre-rotation); see attnfuse_rope."""
    return _rope_call("attnfuse_rope", q, k, out_q, out_k, rope, theta, rope_table)


def attnfuse_rope_bwd(dqr, dkr=None, *, rope="neox", theta=10000.0, out_q=None, out_k=None, rope_table=None):
    """dQ, dK = R^T dQr, R^T dKr; see attnfuse_rope_bwd."""
    return _rope_call("attnfuse_rope_bwd", dqr, dkr, out_q, out_k, rope, theta, rope_table)


def attnfuse_rope_table_bytes(rows, D):
    return _lib.load().attnfuse_rope_table_bytes(rows, D)


def attnfuse_strerror(code):
    return _lib.load().attnfuse_strerror(code).decode()


def attnfuse_version():
    return _lib.load().attnfuse_version()
