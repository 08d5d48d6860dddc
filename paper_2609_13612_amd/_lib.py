"""ctypes loader for lib/libattnfuse.so.

There is no fallback: if the library has not been built this raises, so no
caller can silently run anything but the HIP kernels.
"""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "lib", "libattnfuse.so")

# Signatures of every symbol include/attnfuse.h declares.
_P = ctypes.c_void_p
_I = ctypes.c_int
_F = ctypes.c_float
_L = ctypes.c_longlong
SIGNATURES = {
    "attnfuse_rope_table_bytes": (ctypes.c_size_t, [_I, _I]),
    "attnfuse_rope_table_fill": (_I, [_P, _I, _I, _F, _P]),
    "attnfuse_fwd": (_I, [_P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I, _P, _F, _P]),
    "attnfuse_bwd_workspace_bytes": (ctypes.c_size_t, [_I, _I, _I, _I, _I, _I]),
    "attnfuse_bwd": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                          _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I, _P, _F, _P]),
    "attnfuse_fwd_blocksparse": (_I, [_P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I,
                                      _P, _F, _P]),
    "attnfuse_bwd_blocksparse": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                                      _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I, _P, _F, _P]),
    "attnfuse_fwd_bias_norm": (_I, [_P, _P, _P, _P, _P, _P, _L, _L, _L, _I, _I, _I, _I, _I, _I, _I, _I, _F, _P, _I,
                                    _I, _I, _P, _F, _P]),
    "attnfuse_bwd_bias_norm": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _L, _L, _L, _I, _P, ctypes.c_size_t,
                                    _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I, _P, _F, _P]),
    "attnfuse_rope": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _P]),
    "attnfuse_rope_bwd": (_I, [_P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _P]),
    "attnfuse_decode_workspace_bytes": (ctypes.c_size_t, [_I, _I, _I, _I, _I]),
    "attnfuse_decode": (_I, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t,
                             _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I, _P, _F, _P]),
    "attnfuse_decode_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _F, _P, _I, _I, _I, _P,
                                     _F, _P]),
    "attnfuse_strerror": (ctypes.c_char_p, [_I]),
    "attnfuse_version": (_I, []),
}

_lib = None


def load():
    """The loaded library (cached).  Raises FileNotFoundError if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FileNotFoundError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2609_13612_amd.build` "
                "(there is no non-HIP fallback)")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib
