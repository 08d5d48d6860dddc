"""Pure-Python brute force of RoPE + masked attention, for tiny inputs only.

An independent second formulation used to pin the numpy oracle:
* the rotation is an explicit D x D block-diagonal Givens matrix applied by a
  matrix-vector loop (the oracle rotates pair slices elementwise);
* visibility is decided by explicit comparisons of the key offset i - j;
* softmax, dot products and sums use math.exp / math.fsum over Python floats;
* gradients come from central finite differences of this forward.
"""
import math


def givens_matrix(D, pos, theta, kind):
    """Explicit D x D rotation: a 2x2 block [[c, -s], [s, c]] on each RoPE pair."""
    R = [[1.0 if r == c else 0.0 for c in range(D)] for r in range(D)]
    if kind == "none":
        return R
    half = D // 2
    for i in range(half):
        angle = pos * theta ** (-(2.0 * i) / D)
        c, s = math.cos(angle), math.sin(angle)
        if kind == "neox":
            a, b = i, i + half
        elif kind == "interleaved":
            a, b = 2 * i, 2 * i + 1
        else:
            raise ValueError(kind)
        R[a][a], R[a][b] = c, -s
        R[b][a], R[b][b] = s, c
    return R


def matvec(M, x):
    return [math.fsum(M[r][c] * x[c] for c in range(len(x))) for r in range(len(M))]


def dot(x, y):
    return math.fsum(a * b for a, b in zip(x, y))


def key_visible(i, j, mask, window):
    off = i - j
    if mask == "none":
        return True
    if mask == "causal":
        return off >= 0
    if mask == "sliding_window":
        return 0 <= off < window
    raise ValueError(mask)


def forward(q, k, v, *, rope="none", theta=10000.0, mask="causal", window=None,
            alibi_slopes=None, scale=None, pos_offset=0, block_mask=None, bias=None, norm="softmax"):
    """q: nested lists [B][H][S][D]; k, v: [B][Hkv][S][D]; bias: nested [B][H][S][S] or None.
    Returns (O, LSE) nested lists; under norm="relu" the weights are max(score, 0)
    and LSE is None."""
    B, H, S, D = len(q), len(q[0]), len(q[0][0]), len(q[0][0][0])
    Hkv = len(k[0])
    group = H // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    rot = [givens_matrix(D, p + pos_offset, theta, rope) for p in range(S)]
    O = [[[[0.0] * D for _ in range(S)] for _ in range(H)] for _ in range(B)]
    LSE = [[[0.0] * S for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            kvh = h // group
            for i in range(S):
                qi = matvec(rot[i], q[b][h][i])
                scores = {}
                for j in range(S):
                    if not key_visible(i, j, mask, window):
                        continue
                    if block_mask is not None and not block_mask[1][i // block_mask[0]][j // block_mask[0]]:
                        continue
                    kj = matvec(rot[j], k[b][kvh][j])
                    sc = scale * dot(qi, kj)
                    if alibi_slopes is not None:
                        sc -= alibi_slopes[h] * (i - j)
                    if bias is not None:
                        sc += bias[b][h][i][j]
                    scores[j] = sc
                if norm == "relu":
                    for d in range(D):
                        O[b][h][i][d] = math.fsum(sc * v[b][kvh][j][d] for j, sc in scores.items() if sc > 0.0)
                    continue
                if not scores:
                    LSE[b][h][i] = -math.inf
                    continue
                mx = max(scores.values())
                w = {j: math.exp(sc - mx) for j, sc in scores.items()}
                tot = math.fsum(w.values())
                LSE[b][h][i] = mx + math.log(tot)
                for d in range(D):
                    O[b][h][i][d] = math.fsum(w[j] * v[b][kvh][j][d] for j in w) / tot
    return O, (None if norm == "relu" else LSE)


def loss(q, k, v, do, **kw):
    """sum(O * dO): its gradient w.r.t. q, k, v is the attention backward applied to dO."""
    O, _ = forward(q, k, v, **kw)
    return math.fsum(O[b][h][i][d] * do[b][h][i][d]
                     for b in range(len(O)) for h in range(len(O[0]))
                     for i in range(len(O[0][0])) for d in range(len(O[0][0][0])))


def finite_difference_grad(x, f, eps=1e-6):
    """Central differences of scalar f() w.r.t. every entry of the nested list x (in place)."""
    g = []

    def walk(node, out):
        if isinstance(node[0], list):
            for child in node:
                sub = []
                walk(child, sub)
                out.append(sub)
        else:
            row = []
            for idx in range(len(node)):
                old = node[idx]
                node[idx] = old + eps
                fp = f()
                node[idx] = old - eps
                fm = f()
                node[idx] = old
                row.append((fp - fm) / (2 * eps))
            out.extend(row)

    walk(x, g)
    return g


def decode(q, k_cache, v_cache, cache_lens=None, *, rope="none", theta=10000.0, mask="causal", window=None,
           alibi_slopes=None, scale=None):
    """One query per (b, h) at position len_b - 1 against caches of already-rotated keys.

    q: nested lists [B][H][D]; caches [B][Hkv][S_kv][D].  Returns (O [B][H][D], LSE [B][H]).
    """
    B, H, D = len(q), len(q[0]), len(q[0][0])
    Hkv, S_kv = len(k_cache[0]), len(k_cache[0][0])
    group = H // Hkv
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    lens = [S_kv] * B if cache_lens is None else [int(x) for x in cache_lens]
    O = [[[0.0] * D for _ in range(H)] for _ in range(B)]
    LSE = [[0.0] * H for _ in range(B)]
    for b in range(B):
        p = lens[b] - 1
        rot = givens_matrix(D, p, theta, rope)
        for h in range(H):
            kvh = h // group
            qr = matvec(rot, q[b][h])
            scores = {}
            for j in range(lens[b]):
                if mask == "sliding_window" and not p - j < window:
                    continue
                sc = scale * dot(qr, k_cache[b][kvh][j])
                if alibi_slopes is not None:
                    sc -= alibi_slopes[h] * (p - j)
                scores[j] = sc
            mx = max(scores.values())
            w = {j: math.exp(sc - mx) for j, sc in scores.items()}
            tot = math.fsum(w.values())
            LSE[b][h] = mx + math.log(tot)
            for d in range(D):
                O[b][h][d] = math.fsum(w[j] * v_cache[b][kvh][j][d] for j in w) / tot
    return O, LSE
