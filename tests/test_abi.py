"""The C-ABI library loads without a GPU, exports every declared symbol, and
rejects bad arguments before any HIP call (CPU tests; no compute calls)."""
import ctypes
import os
import re

import pytest

from paper_2609_13612_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attnfuse.h")
FAKE = 0x10000   # aligned, never dereferenced: validation fails first
ODD = 0x10008    # not 16-byte aligned
TABLE = 0x40000  # stand-in for a caller's RoPE cos/sin table


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(attnfuse_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_symbols() == sorted(["attnfuse_bwd", "attnfuse_bwd_bias_norm", "attnfuse_bwd_blocksparse",
                                         "attnfuse_bwd_workspace_bytes", "attnfuse_decode",
                                         "attnfuse_decode_noalloc", "attnfuse_decode_workspace_bytes", "attnfuse_fwd", "attnfuse_fwd_bias_norm",
                                         "attnfuse_fwd_blocksparse", "attnfuse_rope", "attnfuse_rope_bwd",
                                         "attnfuse_rope_table_bytes", "attnfuse_rope_table_fill",
                                         "attnfuse_strerror", "attnfuse_version"])


def test_library_loads_and_exports_every_declared_symbol():
    lib = _lib.load()
    for name in declared_symbols():
        assert hasattr(lib, name), name
    assert set(declared_symbols()) == set(_lib.SIGNATURES)
    assert lib.attnfuse_version() == 3


def test_strerror():
    lib = _lib.load()
    assert lib.attnfuse_strerror(0) == b"success"
    assert b"invalid" in lib.attnfuse_strerror(-1)
    assert b"unsupported" in lib.attnfuse_strerror(-2)
    assert b"HIP" in lib.attnfuse_strerror(-3)
    assert b"static scratch" in lib.attnfuse_strerror(-4)
    assert lib.attnfuse_strerror(7) == b"unknown error code"


def test_workspace_bytes():
    lib = _lib.load()
    rows, krows = 32 * 8192, 8 * 8192
    # delta + lse2 (fp32) + dO (fp16) + dO scale per group (8 x fp32, one
    # 256-byte section) + partial maxima (8 groups x 4*8192*128/16384 = 256
    # chunks x 4 bytes); with RoPE also Q' and K' (fp16)
    scale_parts = 256 + 8 * 256 * 4
    assert lib.attnfuse_bwd_workspace_bytes(1, 32, 8, 8192, 128, 0) == 8 * rows + 2 * rows * 128 + scale_parts
    assert lib.attnfuse_bwd_workspace_bytes(1, 32, 8, 8192, 128, 1) == \
        8 * rows + 2 * rows * 128 * 2 + 2 * krows * 128 + scale_parts
    # sections start on 256-byte boundaries: delta, lse2, dO, scale, maxima, Q', K'
    assert lib.attnfuse_bwd_workspace_bytes(1, 1, 1, 3, 64, 2) == 256 * 2 + 512 + 256 * 2 + 512 * 2
    assert lib.attnfuse_bwd_workspace_bytes(0, 32, 8, 8192, 128, 0) == 0
    assert lib.attnfuse_bwd_workspace_bytes(1, 32, 8, 8192, 128, 7) == 0
    assert lib.attnfuse_bwd_workspace_bytes(1, 6, 4, 8192, 128, 0) == 0   # H % H_kv != 0


def _fwd(**over):
    a = dict(Q=FAKE, K=FAKE + 0x100, V=FAKE + 0x200, O=FAKE + 0x300, LSE=FAKE + 0x400, B=1, H=4, H_kv=2, S=16,
             D=64, dtype=0, rope=1, theta=10000.0, table=TABLE, rows=4096, mask=1, window=0, slopes=None, scale=0.125,
             stream=None)
    a.update(over)
    return _lib.load().attnfuse_fwd(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["H"], a["H_kv"], a["S"],
                                    a["D"], a["dtype"], a["rope"], a["theta"], a["table"], a["rows"], a["mask"],
                                    a["window"], a["slopes"], a["scale"], a["stream"])


INVALID_FWD = [
    dict(Q=None), dict(K=None), dict(V=None), dict(O=None), dict(LSE=None), dict(Q=ODD), dict(LSE=ODD + 0x400),
    dict(O=FAKE), dict(B=0), dict(H=0), dict(H_kv=0), dict(S=0), dict(S=-5), dict(S=(1 << 20) + 1),
    dict(H=3, H_kv=2), dict(D=0), dict(D=63), dict(dtype=2), dict(rope=3), dict(rope=-1),
    dict(theta=0.0), dict(theta=-1.0), dict(theta=float("inf")), dict(theta=float("nan")), dict(mask=3),
    dict(mask=2, window=0), dict(mask=2, window=-4), dict(scale=0.0), dict(scale=-1.0), dict(scale=float("nan")),
    # the caller's RoPE table: present, aligned, covering S, not an output
    dict(table=None), dict(table=ODD), dict(rows=15), dict(rows=0), dict(rows=(1 << 20) + 1),
    dict(table=FAKE + 0x300), dict(table=FAKE + 0x400),
]


@pytest.mark.parametrize("over", INVALID_FWD, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_fwd_rejects_invalid_arguments(over):
    assert _fwd(**over) == -1


@pytest.mark.parametrize("over", [dict(D=96), dict(D=256), dict(D=32), dict(D=96, rope=0)])
def test_fwd_unsupported_head_dim(over):
    assert _fwd(**over) == -2


def test_rope_none_ignores_theta_validation_only_in_attention():
    # theta is irrelevant without RoPE, but D is still checked first for support
    assert _fwd(rope=0, theta=0.0, D=96) == -2


def test_rope_none_needs_no_table():
    # without RoPE the table arguments are ignored (validation passes, D is unsupported)
    assert _fwd(rope=0, table=None, rows=0, D=96) == -2
    assert _fwd(rope=1, table=TABLE, rows=16, D=96) == -2   # exactly S rows is enough


def _bwd(**over):
    base = FAKE
    a = dict(Q=base, K=base + 0x100, V=base + 0x200, O=base + 0x300, dO=base + 0x400, LSE=base + 0x500,
             dQ=base + 0x600, dK=base + 0x700, dV=base + 0x800, ws=base + 0x900, ws_bytes=1 << 20,
             B=1, H=4, H_kv=2, S=16, D=64, dtype=0, rope=1, theta=1e4, table=TABLE, rows=16, mask=1, window=0,
             slopes=None, scale=0.125, stream=None)
    a.update(over)
    return _lib.load().attnfuse_bwd(a["Q"], a["K"], a["V"], a["O"], a["dO"], a["LSE"], a["dQ"], a["dK"], a["dV"],
                                    a["ws"], a["ws_bytes"], a["B"], a["H"], a["H_kv"], a["S"], a["D"], a["dtype"],
                                    a["rope"], a["theta"], a["table"], a["rows"], a["mask"], a["window"],
                                    a["slopes"], a["scale"], a["stream"])


@pytest.mark.parametrize("over", [dict(Q=None), dict(dO=None), dict(ws=None), dict(dQ=FAKE), dict(ws_bytes=20991),
                                  dict(H=4, H_kv=3), dict(mask=2, window=0), dict(dK=ODD), dict(S=0),
                                  dict(table=None), dict(rows=8), dict(table=ODD), dict(table=FAKE + 0x900)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_bwd_rejects_invalid_arguments(over):
    assert _bwd(**over) == -1


def test_bwd_unsupported():
    assert _bwd(D=96) == -2
    assert _bwd(D=96, dtype=1) == -2   # the fp32 debug backward has the same head sizes


def _rope(fn="attnfuse_rope", **over):
    a = dict(Q=FAKE, K=FAKE + 0x100, Qr=FAKE + 0x200, Kr=FAKE + 0x300, B=1, H=4, H_kv=2, S=16, D=64, dtype=0,
             rope=1, theta=1e4, table=TABLE, rows=64, stream=None)
    a.update(over)
    return getattr(_lib.load(), fn)(a["Q"], a["K"], a["Qr"], a["Kr"], a["B"], a["H"], a["H_kv"], a["S"], a["D"],
                                    a["dtype"], a["rope"], a["theta"], a["table"], a["rows"], a["stream"])


@pytest.mark.parametrize("fn", ["attnfuse_rope", "attnfuse_rope_bwd"])
@pytest.mark.parametrize("over", [dict(Q=None), dict(Qr=None), dict(K=None), dict(Kr=None), dict(rope=0),
                                  dict(theta=0.0), dict(H=3), dict(Q=ODD), dict(S=0), dict(dtype=5),
                                  dict(table=None), dict(rows=15), dict(table=FAKE + 0x200), dict(table=FAKE + 0x300)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_rope_rejects_invalid_arguments(fn, over):
    assert _rope(fn, **over) == -1


def test_rope_unsupported():
    assert _rope(D=96) == -2


def test_rope_table_bytes():
    lib = _lib.load()
    assert lib.attnfuse_rope_table_bytes(8192, 128) == 8192 * 64 * 8   # (cos, sin) fp32 per pair
    assert lib.attnfuse_rope_table_bytes(1, 64) == 32 * 8
    assert lib.attnfuse_rope_table_bytes(1 << 20, 128) == (1 << 20) * 64 * 8
    for rows, D in [(0, 128), (-1, 128), ((1 << 20) + 1, 128), (16, 0), (16, 63), (16, -2)]:
        assert lib.attnfuse_rope_table_bytes(rows, D) == 0


@pytest.mark.parametrize("args", [(None, 16, 64, 1e4), (ODD, 16, 64, 1e4), (TABLE, 0, 64, 1e4),
                                  (TABLE, (1 << 20) + 1, 64, 1e4), (TABLE, 16, 63, 1e4), (TABLE, 16, 0, 1e4),
                                  (TABLE, 16, 64, 0.0), (TABLE, 16, 64, -1.0), (TABLE, 16, 64, float("inf")),
                                  (TABLE, 16, 64, float("nan"))], ids=str)
def test_rope_table_fill_rejects_invalid_arguments(args):
    assert _lib.load().attnfuse_rope_table_fill(*args, None) == -1


def test_rope_table_fill_unsupported():
    assert _lib.load().attnfuse_rope_table_fill(TABLE, 16, 96, 1e4, None) == -2


# ----------------------------------------------------------------------------- decode

def test_decode_workspace_bytes():
    lib = _lib.load()
    # Llama-3-70B geometry, 32k cache: 512-key chunks -> 64 per sequence, four
    # wave partials each; 64 heads
    parts = 64 * 64 * 4
    assert lib.attnfuse_decode_workspace_bytes(1, 64, 8, 32768, 128) == parts * 8 + parts * 128 * 4
    # Llama-3-8B geometry, 4k cache: the 128-key minimum -> 32 chunks; 32 heads
    parts = 32 * 32 * 4
    assert lib.attnfuse_decode_workspace_bytes(1, 32, 8, 4096, 128) == parts * 8 + parts * 128 * 4
    # sections start on 256-byte boundaries
    assert lib.attnfuse_decode_workspace_bytes(1, 1, 1, 5, 64) == 256 + 4 * 64 * 4   # 4 partials: 32 B -> 256, 1024
    assert lib.attnfuse_decode_workspace_bytes(0, 32, 8, 4096, 128) == 0
    assert lib.attnfuse_decode_workspace_bytes(1, 6, 4, 4096, 128) == 0
    assert lib.attnfuse_decode_workspace_bytes(1, 32, 8, 0, 128) == 0


def _decode(**over):
    a = dict(Q=FAKE, K=FAKE + 0x100, V=FAKE + 0x200, lens=None, O=FAKE + 0x300, LSE=FAKE + 0x400, ws=FAKE + 0x500,
             ws_bytes=1 << 30, B=2, H=8, H_kv=2, S=300, D=128, dtype=0, rope=1, theta=1e4, table=TABLE, rows=300,
             mask=1, window=0, slopes=None, scale=0.1, stream=None)
    a.update(over)
    return _lib.load().attnfuse_decode(a["Q"], a["K"], a["V"], a["lens"], a["O"], a["LSE"], a["ws"], a["ws_bytes"],
                                       a["B"], a["H"], a["H_kv"], a["S"], a["D"], a["dtype"], a["rope"], a["theta"],
                                       a["table"], a["rows"], a["mask"], a["window"], a["slopes"], a["scale"],
                                       a["stream"])


@pytest.mark.parametrize("over", [dict(Q=None), dict(K=None), dict(V=None), dict(O=None), dict(LSE=None),
                                  dict(ws=None), dict(K=ODD), dict(lens=FAKE + 0x602), dict(O=FAKE),
                                  dict(ws=FAKE + 0x200), dict(ws_bytes=1000), dict(H=8, H_kv=3), dict(S=0),
                                  dict(mask=2, window=0), dict(mask=5), dict(scale=0.0), dict(rope=1, theta=0.0),
                                  dict(dtype=5), dict(table=None), dict(rows=299), dict(table=FAKE + 0x500)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_decode_rejects_invalid_arguments(over):
    assert _decode(**over) == -1


def _decode_na(**over):
    a = dict(Q=FAKE, K=FAKE + 0x100, V=FAKE + 0x200, lens=None, O=FAKE + 0x300, LSE=FAKE + 0x400, B=2, H=8, H_kv=2,
             S=300, D=128, dtype=0, rope=1, theta=1e4, table=TABLE, rows=300, mask=1, window=0, slopes=None,
             scale=0.1, stream=None)
    a.update(over)
    return _lib.load().attnfuse_decode_noalloc(a["Q"], a["K"], a["V"], a["lens"], a["O"], a["LSE"], a["B"], a["H"],
                                               a["H_kv"], a["S"], a["D"], a["dtype"], a["rope"], a["theta"],
                                               a["table"], a["rows"], a["mask"], a["window"], a["slopes"],
                                               a["scale"], a["stream"])


@pytest.mark.parametrize("over", [dict(Q=None), dict(O=None), dict(LSE=None), dict(K=ODD), dict(O=FAKE),
                                  dict(lens=FAKE + 0x602), dict(H=8, H_kv=3), dict(S=0), dict(mask=2, window=0),
                                  dict(scale=0.0), dict(table=None), dict(rows=299), dict(table=FAKE + 0x300)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_decode_noalloc_rejects_invalid_arguments(over):
    assert _decode_na(**over) == -1


def test_decode_noalloc_limits():
    lib = _lib.load()
    assert _decode_na(D=96) == -2 and _decode_na(dtype=1) == -2
    # one sequence, 32 query heads on one K/V head, a 2^20 cache: 512 chunks of
    # 2048 keys, 4 wave partials each, 34 MB of partials > 32 MiB
    big = dict(B=1, H=32, H_kv=1, S=1 << 20, rows=1 << 20)
    assert lib.attnfuse_decode_workspace_bytes(1, 32, 1, 1 << 20, 128) > 32 << 20
    assert _decode_na(**big) == -4
    assert _decode_na(**dict(big, rows=100)) == -1      # argument errors come first


def test_decode_unsupported():
    assert _decode(D=96) == -2
    assert _decode(dtype=1) == -2               # bf16 only
    assert _decode(H=64, H_kv=1) == -2          # more than 32 query heads per K/V head


# ----------------------------------------------------------------------------- block-sparse
MASKP = 0x20000   # 4-byte aligned stand-ins for the device mask lists


def _fwd_bs(**over):
    a = dict(Q=FAKE, K=FAKE + 0x100, V=FAKE + 0x200, O=FAKE + 0x300, LSE=FAKE + 0x400, qp=MASKP, ki=MASKP + 0x100,
             B=1, H=4, H_kv=2, S=16, D=64, dtype=0, rope=1, theta=10000.0, table=TABLE, rows=16, mask=0, window=0,
             slopes=None, scale=0.125, stream=None)
    a.update(over)
    return _lib.load().attnfuse_fwd_blocksparse(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["qp"], a["ki"], a["B"],
                                                a["H"], a["H_kv"], a["S"], a["D"], a["dtype"], a["rope"],
                                                a["theta"], a["table"], a["rows"], a["mask"], a["window"],
                                                a["slopes"], a["scale"], a["stream"])


def _bwd_bs(**over):
    base = FAKE
    a = dict(Q=base, K=base + 0x100, V=base + 0x200, O=base + 0x300, dO=base + 0x400, LSE=base + 0x500,
             dQ=base + 0x600, dK=base + 0x700, dV=base + 0x800, qp=MASKP, ki=MASKP + 0x100, kp=MASKP + 0x200,
             qi=MASKP + 0x300, ws=base + 0x900, ws_bytes=1 << 20, B=1, H=4, H_kv=2, S=16, D=64, dtype=0, rope=1,
             theta=1e4, table=TABLE, rows=16, mask=0, window=0, slopes=None, scale=0.125, stream=None)
    a.update(over)
    return _lib.load().attnfuse_bwd_blocksparse(a["Q"], a["K"], a["V"], a["O"], a["dO"], a["LSE"], a["dQ"], a["dK"],
                                                a["dV"], a["qp"], a["ki"], a["kp"], a["qi"], a["ws"], a["ws_bytes"],
                                                a["B"], a["H"], a["H_kv"], a["S"], a["D"], a["dtype"], a["rope"],
                                                a["theta"], a["table"], a["rows"], a["mask"], a["window"],
                                                a["slopes"], a["scale"], a["stream"])


INVALID_FWD_BS = [dict(qp=None), dict(ki=None), dict(qp=MASKP + 2), dict(ki=MASKP + 0x101), dict(O=MASKP),
                  dict(LSE=MASKP + 0x100), dict(S=64 * 2048 + 1), dict(S=0), dict(Q=None), dict(H=3),
                  dict(mask=2, window=0), dict(scale=0.0), dict(table=None), dict(rows=8)]


@pytest.mark.parametrize("over", INVALID_FWD_BS, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_fwd_blocksparse_rejects_invalid_arguments(over):
    assert _fwd_bs(**over) == -1


def test_fwd_blocksparse_unsupported():
    assert _fwd_bs(D=96) == -2
    assert _fwd_bs(dtype=1) == -2      # bf16 kernels only
    assert _fwd_bs(dtype=1, Q=None) == -1


INVALID_BWD_BS = [dict(qp=None), dict(ki=None), dict(kp=None), dict(qi=None), dict(kp=MASKP + 0x201),
                  dict(dQ=MASKP), dict(ws=MASKP + 0x300), dict(S=64 * 2048 + 1), dict(ws_bytes=100), dict(dO=None),
                  dict(H=4, H_kv=3)]


@pytest.mark.parametrize("over", INVALID_BWD_BS, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_bwd_blocksparse_rejects_invalid_arguments(over):
    assert _bwd_bs(**over) == -1


def test_bwd_blocksparse_unsupported():
    assert _bwd_bs(D=96) == -2
    assert _bwd_bs(dtype=1) == -2


# ----------------------------------------------------------------------------- bias tensor, relu attention
BIASP = 0x30000


def _fwd_bn(**over):
    a = dict(Q=FAKE, K=FAKE + 0x100, V=FAKE + 0x200, O=FAKE + 0x300, LSE=FAKE + 0x400, bias=BIASP, sb=256, sh=64,
             sq=8, norm=0, B=1, H=4, H_kv=2, S=8, D=64, dtype=0, rope=1, theta=10000.0, table=TABLE, rows=8, mask=1,
             window=0, slopes=None, scale=0.125, stream=None)
    a.update(over)
    return _lib.load().attnfuse_fwd_bias_norm(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["bias"], a["sb"], a["sh"],
                                              a["sq"], a["norm"], a["B"], a["H"], a["H_kv"], a["S"], a["D"],
                                              a["dtype"], a["rope"], a["theta"], a["table"], a["rows"], a["mask"],
                                              a["window"], a["slopes"], a["scale"], a["stream"])


def _bwd_bn(**over):
    base = FAKE
    a = dict(Q=base, K=base + 0x100, V=base + 0x200, O=base + 0x300, dO=base + 0x400, LSE=base + 0x500,
             dQ=base + 0x600, dK=base + 0x700, dV=base + 0x800, bias=BIASP, sb=256, sh=64, sq=8, norm=0,
             ws=base + 0x900, ws_bytes=1 << 20, B=1, H=4, H_kv=2, S=8, D=64, dtype=0, rope=1, theta=1e4,
             table=TABLE, rows=8, mask=1, window=0, slopes=None, scale=0.125, stream=None)
    a.update(over)
    return _lib.load().attnfuse_bwd_bias_norm(a["Q"], a["K"], a["V"], a["O"], a["dO"], a["LSE"], a["dQ"], a["dK"],
                                              a["dV"], a["bias"], a["sb"], a["sh"], a["sq"], a["norm"], a["ws"],
                                              a["ws_bytes"], a["B"], a["H"], a["H_kv"], a["S"], a["D"], a["dtype"],
                                              a["rope"], a["theta"], a["table"], a["rows"], a["mask"], a["window"],
                                              a["slopes"], a["scale"], a["stream"])


INVALID_BN = [dict(norm=2), dict(norm=-1), dict(bias=BIASP + 2), dict(sb=-1), dict(sh=-8), dict(sq=-1),
              dict(O=BIASP), dict(Q=None), dict(LSE=None), dict(mask=2, window=0), dict(S=0), dict(table=None),
              dict(rows=7)]


@pytest.mark.parametrize("over", INVALID_BN, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_fwd_bias_norm_rejects_invalid_arguments(over):
    assert _fwd_bn(**over) == -1


def test_fwd_bias_norm_relu_allows_null_lse_only_for_relu():
    assert _fwd_bn(LSE=None, norm=0) == -1
    assert _fwd_bn(LSE=None, norm=1, D=96) == -2     # validation passed; D unsupported


@pytest.mark.parametrize("over", [dict(D=96), dict(dtype=1), dict(slopes=FAKE + 0x1000),
                                  dict(norm=1, dtype=1), dict(norm=1, slopes=FAKE + 0x1000, bias=None)],
                         ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_fwd_bias_norm_unsupported(over):
    assert _fwd_bn(**over) == -2


INVALID_BWD_BN = [dict(norm=3), dict(bias=BIASP + 1), dict(sq=-2), dict(dK=BIASP), dict(ws=BIASP), dict(dO=None),
                  dict(LSE=None), dict(Q=None, LSE=None, norm=1), dict(ws_bytes=10), dict(table=None),
                  dict(table=FAKE + 0x600)]


@pytest.mark.parametrize("over", INVALID_BWD_BN, ids=lambda o: ",".join(f"{k}={v}" for k, v in o.items()))
def test_bwd_bias_norm_rejects_invalid_arguments(over):
    assert _bwd_bn(**over) == -1


def test_bwd_bias_norm_unsupported():
    assert _bwd_bn(D=96) == -2
    assert _bwd_bn(dtype=1) == -2
    assert _bwd_bn(slopes=FAKE + 0x1000) == -2
    assert _bwd_bn(LSE=None, norm=1, D=96) == -2      # LSE is not needed under relu attention


def _declarations():
    """{name: (return type, [parameter types])} parsed from include/attnfuse.h."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    text = re.sub(r"^\s*#[^\n]*", " ", text, flags=re.M)
    out = {}
    for m in re.finditer(r"^\s*((?:const\s+)?\w+(?:\s*\*)?)\s*\b(attnfuse_\w+)\s*\(([^;{]*?)\)\s*;", text, flags=re.M):
        ret, name, params = m.group(1).strip(), m.group(2), m.group(3).strip()
        types = [] if params in ("", "void") else [re.sub(r"\s*\b\w+$", "", p.strip()) for p in params.split(",")]
        out[name] = (ret, types)
    return out


def _ctype_of(c):
    c = " ".join(c.replace("*", " * ").split())
    if c.endswith("*"):
        return ctypes.c_char_p if c in ("const char *",) else ctypes.c_void_p
    return {"int": ctypes.c_int, "float": ctypes.c_float, "size_t": ctypes.c_size_t,
            "long long": ctypes.c_longlong}[c]


def test_binding_signatures_match_the_header():
    """Every ctypes signature the binding declares has the header's parameter
    count and types (pointers as c_void_p), and its return type."""
    decl = _declarations()
    assert set(decl) == set(_lib.SIGNATURES)
    for name, (res, args) in _lib.SIGNATURES.items():
        ret, params = decl[name]
        assert len(args) == len(params), f"{name}: {len(args)} arguments bound, {len(params)} declared"
        for i, (a, pt) in enumerate(zip(args, params)):
            assert a == _ctype_of(pt), f"{name} argument {i}: {pt}"
        assert res == _ctype_of(ret), f"{name}: return type {ret}"
