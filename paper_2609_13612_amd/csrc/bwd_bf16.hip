// Fused RoPE + masked attention backward, bf16 MFMA with fp32 accumulation,
// for gfx950.
//
// The passes of Section 4.4, no atomics: every output tile has exactly one
// writer.
//   0. bwd_dmax, bwd_dscale: sigma, the power of two per (batch, K/V head)
//                 that brings the group's largest |dO| into [1, 2).
//   1. bwd_prep:  delta_i = rowsum(dO_i * O_i), LSE_i in log2 units, sigma dO
//                 in fp16, and with RoPE Q' = R Q and K' = R K rotated once
//                 into the workspace (fp16).  The later kernels read each Q'
//                 and K' tile many times (dK/dV reads every Q' tile once per
//                 key block), so one rotation pass replaces all of those.
//   2. bwd_dq:    one workgroup per 256 query rows (GQA heads packed, as in
//                 the forward); it loops over visible key tiles:
//                 dQ' += scale dS K',  dQ = R^T dQ'.  Since it forms P and dP
//                 for every visible key of its rows, it also sums the
//                 softmax backward's row term delta_i = sum_j P_ij dP_ij in
//                 fp32 (with P renormalised by its own row sum) and writes it,
//                 and the renormalised LSE, over the preprocessing pass's.
//   3. bwd_dkdv:  one workgroup per 128 keys of one (batch, K/V head); it
//                 loops over the query heads of the GQA group and their
//                 visible query tiles, re-deriving P = exp(S - LSE) tile by
//                 tile:  dV += P^T dO,  dS = P o (dO V^T - delta),
//                 dK' += scale dS^T Q';  dK = R^T dK'.
// delta from rowsum(dO o O) equals sum_j P_ij dP_ij only for the exact O;
// the bf16 O a forward stores moves it by O's rounding, which reaches dK and
// dQ through P_ij (dP_ij - delta_i).  The dK/dV pass therefore runs last, on
// the dQ pass's sum; the dQ pass itself uses the preprocessing pass's value.
//
// Scaling: the fp16 MFMA operands dO and dS carry the factor sigma, so their
// magnitudes sit near 1 whatever the gradient's scale (unscaled bf16
// gradients of 1e-6 would fall into fp16's subnormals, 6e-8 apart); the
// gradients leave multiplied by 1/sigma.  Multiplying by a power of two is
// exact, so results do not depend on the scale of dO.
// Register layouts follow the forward: the operand held in registers is the
// MFMA B operand (lane = its row), tiles staged in LDS are the A operand, and
// contractions over queries/keys read a transposed LDS copy stored with the
// perm16 row order that matches the score tile's register order.
//
// Precision: Q', K' and dS are fp16 MFMA operands.  With RoPE the rotated
// Q' and K' are the fp16 values the forward's scores came from, so P is
// re-derived from the same rounded operands that produced its LSE; without
// RoPE, Q and K are converted exactly from bf16 as they are staged.  dS in
// fp16 (2^-12 relative rounding instead of bf16's 2^-9) keeps the sums
// dK = dS^T Q and dQ = dS K accurate when attention concentrates on a few
// keys and their gradients grow.  dV = P^T dO sums P over many queries
// without normalisation, so it also runs on fp16 operands (P and sigma dO,
// the latter converted exactly from bf16).  Range: the rotated |Q'|, |K'|
// and |V| must stay below the fp16 maximum 65504, and |sigma dS| <= 4 D
// max|V| below it too, i.e. max|V| < 16376 / D (128 at D = 128).  In the dQ
// pass dP = dO V^T uses the bf16 inputs as they are.
#include <type_traits>

#include "attn_tiles.hpp"
#include "launch.hpp"

namespace af {

// ---------------------------------------------------------------- dO scale
// Partial maxima of |dO| over chunks of each (batch, K/V head)'s G query heads
// (contiguous in [B, H, S, D]), as bf16 magnitude bits: the bit patterns of
// non-negative bf16 values order like the values, so the maximum is an
// integer maximum.
constexpr int DMAX_CHUNK = 16384;   // dO elements per partial maximum

template <int D>
__global__ __launch_bounds__(256) void bwd_dmax_kernel(BwdParams p) {
  const int nch = p.dmax_chunks;
  const int bg = blockIdx.x / nch, c = blockIdx.x - bg * nch;
  const long long n = (long long)(p.H / p.Hkv) * p.S * D;
  const uint16_t* src = static_cast<const uint16_t*>(p.dout) + (long long)bg * n;
  const long long e1 = min(n, (long long)(c + 1) * DMAX_CHUNK);
  uint32_t mx = 0;
  for (long long e = (long long)c * DMAX_CHUNK + 8 * threadIdx.x; e < e1; e += 8 * 256) {   // n % 8 == 0
    const u32x4 x = ld16(src + e);
#pragma unroll
    for (int w = 0; w < 4; ++w) mx = max(mx, max(x[w] & 0x7fffu, (x[w] >> 16) & 0x7fffu));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, 64));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) p.dmax[blockIdx.x] = max(max(part[0], part[1]), max(part[2], part[3]));
}

// sigma = 2^(127 - E) for the largest |dO| with biased exponent E, so that
// max |dO| * sigma lies in [1, 2); clamped to [2^-126, 2^126].  1 when the
// group's dO is all zero or holds an inf / NaN.  One workgroup per group.
__global__ __launch_bounds__(256) void bwd_dscale_kernel(BwdParams p) {
  const int bg = blockIdx.x, nch = p.dmax_chunks;
  uint32_t mx = 0;
  for (int c = threadIdx.x; c < nch; c += 256) mx = max(mx, p.dmax[(long long)bg * nch + c]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = max(mx, (uint32_t)__shfl_xor((int)mx, off, 64));
  __shared__ uint32_t part[4];
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = mx;
  __syncthreads();
  if (threadIdx.x == 0) {
    mx = max(max(part[0], part[1]), max(part[2], part[3]));
    const int E = (int)(mx >> 7);   // bf16 biased exponent (the sign bit is clear)
    float sig = 1.f;
    if (mx != 0u && E != 255) sig = __uint_as_float((uint32_t)min(max(254 - max(E, 1), 1), 253) << 23);
    p.dscale[bg] = sig;
  }
}

// ---------------------------------------------------------------- preprocessing
// One thread per (row, chunk pair c): chunks c and c + D/16 (dims 8c.. and
// D/2 + 8c..), which are NeoX partners; interleaved pairs stay in-chunk.
// Blocks [0, q_blocks) cover the B*H query rows, the rest the B*H_kv key rows.
template <int D, int ROPE>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdParams p, int q_blocks) {
  constexpr int TPR = D / 16;            // threads per row
  constexpr int RPB = 256 / TPR;         // rows per block
  const int c = threadIdx.x % TPR;
  const int d0 = 8 * c, d1 = D / 2 + 8 * c;
  if ((int)blockIdx.x < q_blocks) {
    const long long rows = (long long)p.B * p.H * p.S;
    const long long row = (long long)blockIdx.x * RPB + threadIdx.x / TPR;
    const long long rc = row < rows ? row : rows - 1;   // clamp: every lane joins the reduction
    const int hq = (int)((rc / p.S) % p.H), bq = (int)(rc / ((long long)p.S * p.H));
    const float sig = p.dscale[bq * p.Hkv + hq / (p.H / p.Hkv)];
    const uint16_t* dOr = static_cast<const uint16_t*>(p.dout) + rc * D;
    const uint16_t* Or = static_cast<const uint16_t*>(p.o) + rc * D;
    const u32x4 a0 = ld16(dOr + d0), a1 = ld16(dOr + d1);
    const u32x4 o0 = ld16(Or + d0), o1 = ld16(Or + d1);
    float acc = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w)
      acc += bf_lo(a0[w]) * bf_lo(o0[w]) + bf_hi(a0[w]) * bf_hi(o0[w]) + bf_lo(a1[w]) * bf_lo(o1[w]) +
             bf_hi(a1[w]) * bf_hi(o1[w]);
#pragma unroll
    for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, TPR);
    if (row < rows) {
      u32x4 h0, h1;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        h0[w] = pack_f16(bf_lo(a0[w]) * sig, bf_hi(a0[w]) * sig);
        h1[w] = pack_f16(bf_lo(a1[w]) * sig, bf_hi(a1[w]) * sig);
      }
      uint16_t* dst = static_cast<uint16_t*>(p.do16) + row * D;
      st16(dst + d0, h0);
      st16(dst + d1, h1);
      if (c == 0) {
        p.delta[row] = acc * sig;
        const float l = p.lse ? p.lse[row] : 0.f;   // relu attention has no LSE
        p.lse2[row] = (l == -INFINITY) ? INFINITY : l * kLog2e;
      }
      if constexpr (ROPE != ROPE_NONE) {
        const int pos = (int)(row % p.S);
        const uint16_t* Qr = static_cast<const uint16_t*>(p.q) + row * D;
        u32x4 q0 = ld16(Qr + d0), q1 = ld16(Qr + d1);
        if constexpr (ROPE == ROPE_NEOX) {
          rotate_neox8<false, true>(q0, q1, p.table + (size_t)pos * (D / 2) + 8 * c);
        } else {
          rotate_interleaved8<false, true>(q0, p.table + (size_t)pos * (D / 2) + 4 * c);
          rotate_interleaved8<false, true>(q1, p.table + (size_t)pos * (D / 2) + D / 4 + 4 * c);
        }
        uint16_t* qd = static_cast<uint16_t*>(p.qr16) + row * D;
        st16(qd + d0, q0);
        st16(qd + d1, q1);
      }
    }
  } else if constexpr (ROPE != ROPE_NONE) {
    const long long rows = (long long)p.B * p.Hkv * p.S;
    const long long row = (long long)(blockIdx.x - q_blocks) * RPB + threadIdx.x / TPR;
    if (row < rows) {
      const int pos = (int)(row % p.S);
      const uint16_t* Kr = static_cast<const uint16_t*>(p.k) + row * D;
      u32x4 k0 = ld16(Kr + d0), k1 = ld16(Kr + d1);
      if constexpr (ROPE == ROPE_NEOX) {
        rotate_neox8<false, true>(k0, k1, p.table + (size_t)pos * (D / 2) + 8 * c);
      } else {
        rotate_interleaved8<false, true>(k0, p.table + (size_t)pos * (D / 2) + 4 * c);
        rotate_interleaved8<false, true>(k1, p.table + (size_t)pos * (D / 2) + D / 4 + 4 * c);
      }
      uint16_t* kd = static_cast<uint16_t*>(p.kr16) + row * D;
      st16(kd + d0, k0);
      st16(kd + d1, k1);
    }
  }
}

// ---------------------------------------------------------------- helpers
// Load one lane's row of a bf16 matrix as the MFMA B operand (dims 16s + 8lg..+7),
// RoPE-rotated in-lane (rotated values rounded to fp16) or, with TO_F16,
// converted to fp16 unrotated.  Rows >= S give zeros.
template <int D, int ROPE, bool TO_F16 = false>
__device__ __forceinline__ void load_row_operand(u32x4 (&reg)[D / 16], const uint16_t* __restrict__ src,
                                                 const float2* __restrict__ table, int n, int S, int lg) {
  constexpr int KS = D / 16;
#pragma unroll
  for (int s = 0; s < KS; ++s) reg[s] = (n < S) ? ld16(src + (size_t)n * D + 16 * s + 8 * lg) : u32x4{0, 0, 0, 0};
  if (n < S) {
    if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
      for (int s = 0; s < KS / 2; ++s)
        rotate_neox8<false, true>(reg[s], reg[s + KS / 2], table + (size_t)n * (D / 2) + 16 * s + 8 * lg);
    } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
      for (int s = 0; s < KS; ++s) rotate_interleaved8<false, true>(reg[s], table + (size_t)n * (D / 2) + 8 * s + 4 * lg);
    }
  }
  if constexpr (TO_F16 && ROPE == ROPE_NONE) {
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int w = 0; w < 4; ++w) reg[s][w] = pack_f16(bf_lo(reg[s][w]), bf_hi(reg[s][w]));
  }
}

// Scale, undo the rotation and store an accumulator tile X^T (d x rows) whose
// lane owns row n: element r of tile mt is dim 32 mt + 8 (r/4) + 4 lg + r%4.
template <int D, int ROPE>
__device__ __forceinline__ void store_grad_rows(f32x16 (&acc)[D / 32], float scale, uint16_t* __restrict__ dst,
                                                const float2* __restrict__ table, int n0, int S,
                                                uint16_t* __restrict__ lds, int lane) {
  constexpr int MT = D / 32;
  const int lg = lane >> 5, n = min(n0 + (lane & 31), S - 1);   // this lane's row (rows past S: not stored)
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) acc[mt] *= scale;
  if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
    for (int mt = 0; mt < MT / 2; ++mt) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const float4* t = reinterpret_cast<const float4*>(table + (size_t)n * (D / 2) + 32 * mt + 8 * a + 4 * lg);
        const float4 t0 = t[0], t1 = t[1];
        const float cs[4][2] = {{t0.x, t0.y}, {t0.z, t0.w}, {t1.x, t1.y}, {t1.z, t1.w}};
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          float xa = acc[mt][4 * a + b], xb = acc[mt + MT / 2][4 * a + b];
          rotate_pair<true>(xa, xb, cs[b][0], cs[b][1]);
          acc[mt][4 * a + b] = xa;
          acc[mt + MT / 2][4 * a + b] = xb;
        }
      }
    }
  } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const float4 t = *reinterpret_cast<const float4*>(table + (size_t)n * (D / 2) + 16 * mt + 4 * a + 2 * lg);
        float x0 = acc[mt][4 * a + 0], x1 = acc[mt][4 * a + 1], x2 = acc[mt][4 * a + 2], x3 = acc[mt][4 * a + 3];
        rotate_pair<true>(x0, x1, t.x, t.y);
        rotate_pair<true>(x2, x3, t.z, t.w);
        acc[mt][4 * a + 0] = x0;
        acc[mt][4 * a + 1] = x1;
        acc[mt][4 * a + 2] = x2;
        acc[mt][4 * a + 3] = x3;
      }
    }
  }
  store_rows_bf16<D>(acc, lds, dst + (size_t)n0 * D, S - n0, lane);
}

// Transposed MFMA A operand from a row-major LDS tile: rows (keys or queries)
// base_row + {4 lg + i/4, +8} and 16 dims per 16-lane group (lds_read_tr16).
__device__ __forceinline__ u32x4 tr_operand(const uint16_t* tile, int pitch, int row0, int col0, int lane) {
  const int lg = lane >> 5;
  const uint16_t* p = tile + (row0 + 4 * lg + ((lane & 15) >> 2)) * pitch + col0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const u32x2 lo = lds_read_tr16(p);
  const u32x2 hi = lds_read_tr16(p + 8 * pitch);
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// The same operand from a swizzled tile (swz_at): rows row0 + {4 lg + i/4, +8}
// (row0 a multiple of 16), columns 32 mt + ..., through the lane's SwzLane.
template <int D>
__device__ __forceinline__ u32x4 tr_operand_swz(const uint16_t* tile, const SwzLane<D>& z, int row0, int mt) {
  const uint16_t* t = tile + row0 * D;
  const u32x2 lo = lds_read_tr16(t + (z.tr_base[0] ^ (32 * mt)));
  const u32x2 hi = lds_read_tr16(t + (z.tr_base[1] ^ (32 * mt)));
  return u32x4{lo[0], lo[1], hi[0], hi[1]};
}

// A row operand (lane = row row0 + l % 32, k-step k) from a swizzled tile.
template <int D>
__device__ __forceinline__ u32x4 row_operand_swz(const uint16_t* tile, const SwzLane<D>& z, int row0, int k) {
  return *reinterpret_cast<const u32x4*>(tile + row0 * D + (z.row_base ^ (16 * k)));
}

// ---------------------------------------------------------------- dK / dV
// Query-side tile of the dK/dV kernel: BQ_ query rows of Q' (fp16, rotated by
// the preprocessing kernel) or Q (bf16, converted to fp16 as it is staged)
// and of dO (fp16), plus their LSE (log2 units) and delta.
template <int D, int BQ_ = 64>
struct QTileCfg {
  static constexpr int NW = 8;                // two waves per SIMD
  static constexpr int THREADS = 64 * NW;
  static constexpr int KEYS = 32 * NW / 2;    // keys per workgroup: each 32 keys are shared by a wave pair
  static constexpr int BQ = BQ_;              // query rows per tile: the pair splits them in halves
  static constexpr int VP = D + 8;            // pitch of the resident K' and V rows (16-byte reads)
  static constexpr int V_ELEMS = KEYS * VP;
  static constexpr int KS = D / 16;
  static constexpr int MT = D / 32;
  static constexpr int Q_ELEMS = BQ * D;      // Q' and dO tiles: read by rows and transposed, so swizzled (swz_at)
  static constexpr int STAGE = 2 * Q_ELEMS;   // Q' then dO
  static constexpr int ITEMS = BQ * (D / 8);  // 16-byte chunks per matrix
  static constexpr int IPT = (ITEMS + THREADS - 1) / THREADS;
};

template <int D, int BQ = 64>
struct QTileRegs {
  using C = QTileCfg<D, BQ>;
  u32x4 q[C::IPT];
  u32x4 o[C::IPT];
  float lse2, del;
};

// Rows past S are clamped to row S-1 so every load is unconditional; they get
// LSE = +inf (so P = 0) and delta = 0, so they contribute nothing.
template <int D, int BQ>
__device__ __forceinline__ void qtile_load(QTileRegs<D, BQ>& R, const uint16_t* __restrict__ Q,
                                           const uint16_t* __restrict__ dO, const float* __restrict__ lse2,
                                           const float* __restrict__ delta, int m0, int S, int tid) {
  using C = QTileCfg<D, BQ>;
#pragma unroll
  for (int i = 0; i < C::IPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::ITEMS % C::THREADS != 0 && it >= C::ITEMS) break;
    const int r = it / (D / 8), c = it % (D / 8), m = min(m0 + r, S - 1);
    R.q[i] = ld16(Q + (size_t)m * D + 8 * c);
    R.o[i] = ld16(dO + (size_t)m * D + 8 * c);
  }
  const int ms = min(m0 + (tid & (C::BQ - 1)), S - 1);
  const bool in = m0 + (tid & (C::BQ - 1)) < S;
  const float l = lse2[ms], dl = delta[ms];
  R.lse2 = in ? l : INFINITY;
  R.del = in ? dl : 0.f;
}

// TO_F16: Q arrives as bf16 (no RoPE) and is converted as it is staged.
template <int D, bool TO_F16, int BQ>
__device__ __forceinline__ void qtile_commit(const QTileRegs<D, BQ>& R, uint16_t* __restrict__ Qs,
                                             uint16_t* __restrict__ Os, float* __restrict__ lse2s,
                                             float* __restrict__ dels, int tid) {
  using C = QTileCfg<D, BQ>;
#pragma unroll
  for (int i = 0; i < C::IPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::ITEMS % C::THREADS != 0 && it >= C::ITEMS) break;
    const int r = it / (D / 8), c = it % (D / 8);
    u32x4 q = R.q[i];
    if constexpr (TO_F16) {
#pragma unroll
      for (int w = 0; w < 4; ++w) q[w] = pack_f16(bf_lo(q[w]), bf_hi(q[w]));
    }
    *reinterpret_cast<u32x4*>(Qs + swz_at<D>(r, 8 * c)) = q;
    *reinterpret_cast<u32x4*>(Os + swz_at<D>(r, 8 * c)) = R.o[i];
  }
  if (tid < C::BQ) {
    lse2s[tid] = R.lse2;
    dels[tid] = R.del;
  }
}

// One workgroup = 8 waves = 128 keys of one (batch, K/V head).  Waves w and
// w + 4 share keys 32 (w % 4) .. +31 and split every query tile (64 rows;
// 128 at D = 64 without a block mask), w taking its first half and w + 4 the
// second, 32 rows at a time, so two waves per SIMD hide each other's
// latencies; their partial dK/dV are summed through LDS at the end.
// The block's K' rows (B operand of S = Q' K'^T) and V rows (fp16, B operand
// of dP = dO V^T) stay resident in LDS, leaving the registers to the dK/dV
// accumulators.
template <int D, int ROPE, int MASK, bool ALIBI, bool SPARSE, int EXT = EXT_NONE>
__global__ __launch_bounds__(512) void bwd_dkdv_kernel(BwdParams p) {
  // at D = 64 a 128-row query tile halves the steps (barriers, staging) per
  // key block; block masks work in 64-row blocks
  using C = QTileCfg<D, (D == 64 && !SPARSE) ? 128 : 64>;
  constexpr int NQ = C::BQ / 64;   // 32-row blocks of a tile per wave
  constexpr bool TBIAS = EXT == EXT_BIAS || EXT == EXT_RELU_BIAS;
  constexpr bool RELU = EXT == EXT_RELU || EXT == EXT_RELU_BIAS;
  constexpr bool ROT = ROPE != ROPE_NONE;    // Q' and K' come rotated (fp16) from the workspace
  constexpr int SMEM = 2 * C::STAGE + 2 * C::V_ELEMS;
  static_assert(SMEM * 2 >= 4 * 16 * C::MT * 64 * 4, "the partial-sum exchange reuses the staging memory");
  __shared__ __attribute__((aligned(16))) uint16_t smem[SMEM];
  __shared__ __attribute__((aligned(16))) float stat[2][2][C::BQ];   // [stage][lse2, delta][query]
  uint16_t* Ks = smem + 2 * C::STAGE;
  uint16_t* Vs = Ks + C::V_ELEMS;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, lq = lane & 31, lg = lane >> 5;
  const int kw = wave & 3, qh = wave >> 2;    // key block within the workgroup, query half
  const int S = p.S;
  const int BG = p.B * p.Hkv;
  const int bg = blockIdx.x % BG;
  const int kb = (int)(blockIdx.x / BG);   // ascending: under a causal mask the first key blocks see the most queries
  const int b = bg / p.Hkv, g = bg % p.Hkv;
  const int G = p.H / p.Hkv;
  const int nb = kb * C::KEYS;        // first key of the block
  const int nw = nb + 32 * kw;        // first key of this wave
  const int n = nw + lq;              // this lane's key

  // K' (fp16, rotated by the preprocessing kernel) or K (bf16) as is, and V
  // converted to fp16; rows past S clamped (their results are not stored)
  const uint16_t* Kg = static_cast<const uint16_t*>(ROT ? p.kr16 : p.k) + (size_t)bg * S * D;
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v) + (size_t)bg * S * D;
  constexpr int VITEMS = C::KEYS * (D / 8);
#pragma unroll
  for (int i = 0; i < VITEMS / C::THREADS; ++i) {
    const int it = tid + C::THREADS * i;
    const int r = it / (D / 8), c = it % (D / 8);
    const size_t off = (size_t)min(nb + r, S - 1) * D + 8 * c;
    u32x4 v = ld16(Vg + off);
    u32x4 k = ld16(Kg + off);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      v[w] = pack_f16(bf_lo(v[w]), bf_hi(v[w]));
      if constexpr (!ROT) k[w] = pack_f16(bf_lo(k[w]), bf_hi(k[w]));
    }
    *reinterpret_cast<u32x4*>(Vs + r * C::VP + 8 * c) = v;
    *reinterpret_cast<u32x4*>(Ks + r * C::VP + 8 * c) = k;
  }

  f32x16 dk[C::MT], dv[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) { dk[i] = f32x16{}; dv[i] = f32x16{}; }

  const float c2 = p.scale * kLog2e;
  const int W = p.window;
  const int ntq = (S + C::BQ - 1) / C::BQ;
  int tq_begin = 0, tq_end = ntq;
  if constexpr (MASK != MASK_NONE) tq_begin = nb / C::BQ;
  if constexpr (MASK == MASK_SLIDING_WINDOW) tq_end = min(ntq, (min(nb + C::KEYS - 1, S - 1) + W - 1) / C::BQ + 1);
  // Query tiles by position: tq_begin + i, or under a block-sparse mask the
  // union of the active query blocks of the workgroup's two 64-key blocks
  // (the mask by key block), with a bit per key block saying which hold it.
  __shared__ std::conditional_t<SPARSE, TileList<true>, int> tl;
  int nq = max(0, tq_end - tq_begin);
  const int jw = kw >> 1;             // this wave's 64-key block within the workgroup
  if constexpr (SPARSE) {             // the query staging memory serves as scratch: nothing is staged yet
    const int r0 = nb / C::BQ, r1 = (min(nb + C::KEYS, S) - 1) / C::BQ;
    nq = __builtin_amdgcn_readfirstlane(build_tile_list<C::THREADS>(tl, smem, p.bk_ptr, p.bq_idx, r0, r1 - r0 + 1,
                                                                    ntq, tq_begin, tq_end, tid));
  }
  const int steps = G * nq;           // (query head of the group, query tile) pairs

  auto head_of = [&](int s) { return g * G + s / nq; };
  auto tile_of = [&](int s) -> int {
    if constexpr (SPARSE) return __builtin_amdgcn_readfirstlane((int)tl.tile[s % nq]);
    else return tq_begin + s % nq;
  };
  auto src = [&](int s, const uint16_t*& Qh, const uint16_t*& dOh, const float*& l2, const float*& dl) {
    const size_t bh = (size_t)b * p.H + head_of(s);
    Qh = static_cast<const uint16_t*>(ROT ? p.qr16 : p.q) + bh * S * D;
    dOh = static_cast<const uint16_t*>(p.do16) + bh * S * D;
    l2 = p.lse2 + bh * S;
    dl = p.delta + bh * S;
  };

  QTileRegs<D, C::BQ> R;
  if (steps > 0) {
    const uint16_t *Qh, *dOh;
    const float *l2, *dl;
    src(0, Qh, dOh, l2, dl);
    qtile_load<D>(R, Qh, dOh, l2, dl, tile_of(0) * C::BQ, S, tid);
    qtile_commit<D, !ROT>(R, smem, smem + C::Q_ELEMS, stat[0][0], stat[0][1], tid);
  }
  __syncthreads();

  const SwzLane<D> zl(lane);
  for (int s = 0; s < steps; ++s) {
    const int st = s & 1;
    const SwzLane<D> z = zl.opaque();
    const uint16_t* Qs = smem + st * C::STAGE;
    const uint16_t* Os = Qs + C::Q_ELEMS;
    const float* lse2s = stat[st][0];
    const float* dels = stat[st][1];
    const bool more = s + 1 < steps;
    if (more) {
      const uint16_t *Qh, *dOh;
      const float *l2, *dl;
      src(s + 1, Qh, dOh, l2, dl);
      qtile_load<D>(R, Qh, dOh, l2, dl, tile_of(s + 1) * C::BQ, S, tid);
    }
    const int h = head_of(s);
    const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;
    const float* __restrict__ bcol = nullptr;      // this lane's key column of the bias tensor
    if constexpr (TBIAS) bcol = p.bias + b * p.bias_sb + h * p.bias_sh + min(n, S - 1);
#pragma unroll
    for (int j = 0; j < NQ; ++j) {
      const int qt = NQ * qh + j;                  // this wave's 32-row block of the tile
      const int mq = tile_of(s) * C::BQ + 32 * qt;   // its first query row

      bool visible = nw < S;
      if constexpr (SPARSE) visible = visible && ((tl.rows[s % nq] >> jw) & 1);
      if constexpr (MASK != MASK_NONE) visible = visible && (mq + 31 >= nw);
      if constexpr (MASK == MASK_SLIDING_WINDOW) visible = visible && (mq <= nw + 31 + W - 1);
      if (visible) {
        bool need_mask = nw + 32 > S;
        if constexpr (RELU) need_mask = need_mask || (mq + 32 > S);   // no LSE zeroes the rows past S
        if constexpr (MASK != MASK_NONE) need_mask = need_mask || (mq < nw + 31);
        if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (mq + 31 - W >= nw);
        // S = Q' K'^T and dP = dO V^T for 32 queries (rows) x this wave's 32 keys
        // (columns); the two MFMA chains are interleaved.
        f32x16 sc = f32x16{}, dp = f32x16{};
  #pragma unroll
        for (int k = 0; k < C::KS; ++k) {
          const u32x4 aq = row_operand_swz<D>(Qs, z, 32 * qt, k);
          const u32x4 ao = row_operand_swz<D>(Os, z, 32 * qt, k);
          const u32x4 bk = *reinterpret_cast<const u32x4*>(Ks + (32 * kw + lq) * C::VP + 16 * k + 8 * lg);
          const u32x4 bv = *reinterpret_cast<const u32x4*>(Vs + (32 * kw + lq) * C::VP + 16 * k + 8 * lg);
          sc = mfma32<true>(aq, bk, sc);
          dp = mfma32<true>(ao, bv, dp);
        }
        // element r: query mq + 8 (r/4) + 4 lg + r%4, key n
        float pr[16], ds[16];
        float bias[16] = {};   // the bias column of key n at the 16 rows
        if constexpr (TBIAS) {
          if (p.bias_sq == 0) {   // broadcast over queries (e.g. key padding): one value
            const float b0 = bcol[0];
  #pragma unroll
            for (int r = 0; r < 16; ++r) bias[r] = b0;
          } else {
  #pragma unroll
            for (int r = 0; r < 16; ++r)
              bias[r] = bcol[(long long)min(mq + 8 * (r >> 2) + 4 * lg + (r & 3), S - 1) * p.bias_sq];
          }
        }
  #pragma unroll
        for (int a = 0; a < 4; ++a) {
          const int qlb = 32 * qt + 8 * a + 4 * lg;
          const float4 l4 = *reinterpret_cast<const float4*>(lse2s + qlb);
          const float4 d4 = *reinterpret_cast<const float4*>(dels + qlb);
          const float lv[4] = {l4.x, l4.y, l4.z, l4.w};
          const float dv4[4] = {d4.x, d4.y, d4.z, d4.w};
  #pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = 4 * a + e;
            if constexpr (TBIAS || RELU) {
              const float bv = bias[r];
              if constexpr (RELU) {   // P = max(s, 0), dS = dP where s > 0
                const float x = __builtin_fmaf(sc[r], p.scale, bv);
                pr[r] = fmaxf(x, 0.f);
                ds[r] = (x > 0.f) ? dp[r] : 0.f;
              } else {
                pr[r] = fast_exp2(__builtin_fmaf(sc[r], c2, bv * kLog2e) - lv[e]);
                ds[r] = dp[r] - dv4[e];
              }
            } else {
              const float x = ALIBI ? __builtin_fmaf(sc[r], c2, slope2 * (float)(n - (mq + 8 * a + 4 * lg + e))) : sc[r] * c2;
              pr[r] = fast_exp2(x - lv[e]);
              ds[r] = dp[r] - dv4[e];
            }
          }
        }
        if (need_mask) {   // wave-uniform: diagonal, window-edge and sequence-end tiles only
  #pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int m = mq + 8 * (r >> 2) + 4 * lg + (r & 3);
            bool ok = n < S;
            if constexpr (RELU) ok = ok && (m < S);
            if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
            if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
            pr[r] = ok ? pr[r] : 0.f;
            if constexpr (RELU) ds[r] = ok ? ds[r] : 0.f;
          }
        }
        if constexpr (!RELU) {
  #pragma unroll
          for (int r = 0; r < 16; ++r) ds[r] *= pr[r];
        }
        u32x4 pb[2], db[2];
  #pragma unroll
        for (int hf = 0; hf < 2; ++hf)
  #pragma unroll
          for (int w = 0; w < 4; ++w) {
            pb[hf][w] = pack_f16(pr[8 * hf + 2 * w], pr[8 * hf + 2 * w + 1]);
            db[hf][w] = pack_f16(ds[8 * hf + 2 * w], ds[8 * hf + 2 * w + 1]);
          }
        // dV^T += dO^T P and dK'^T += Q'^T dS (transposed operands from row-major
        // tiles).  The next pair's operands are read before this pair's MFMAs, so
        // each MFMA waits on a read issued one pair earlier rather than on its own.
        {
          constexpr int NI = 2 * C::MT;   // (hf, mt) pairs
          u32x4 to = tr_operand_swz<D>(Os, z, 32 * qt, 0), tq = tr_operand_swz<D>(Qs, z, 32 * qt, 0);
  #pragma unroll
          for (int i = 0; i < NI; ++i) {
            const int hf = i / C::MT, mt = i % C::MT;
            const u32x4 ao = to, aq = tq;
            if (i + 1 < NI) {
              const int row = 32 * qt + 16 * ((i + 1) / C::MT), mn = (i + 1) % C::MT;
              to = tr_operand_swz<D>(Os, z, row, mn);
              tq = tr_operand_swz<D>(Qs, z, row, mn);
            }
            dv[mt] = mfma32<true>(ao, pb[hf], dv[mt]);
            dk[mt] = mfma32<true>(aq, db[hf], dk[mt]);
          }
        }
      }
    }

    if (more) {
      const int sn = (s + 1) & 1;
      qtile_commit<D, !ROT>(R, smem + sn * C::STAGE, smem + sn * C::STAGE + C::Q_ELEMS, stat[sn][0], stat[sn][1], tid);
    }
    __syncthreads();
  }

  // Sum the pair's partials: the second wave of a pair hands over its dK, the
  // first its dV, through [key block][element][lane] in the staging memory.
  float* xch = reinterpret_cast<float*>(smem);
  auto put = [&](f32x16 (&x)[C::MT]) {
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) xch[(kw * (16 * C::MT) + 16 * mt + r) * 64 + lane] = x[mt][r];
  };
  auto add = [&](f32x16 (&x)[C::MT]) {
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int r = 0; r < 16; ++r) x[mt][r] += xch[(kw * (16 * C::MT) + 16 * mt + r) * 64 + lane];
  };
  if (qh == 1) put(dk);
  __syncthreads();
  if (qh == 0) add(dk);
  __syncthreads();
  if (qh == 0) put(dv);
  __syncthreads();
  if (qh == 1) add(dv);
  __syncthreads();   // the exchange memory is free again: each wave's output rows go through it

  {   // dS and dO carried the factor sigma (a power of two: exact)
    static_assert(C::THREADS / 64 * OUT_ROWS_ELEMS<D> <= SMEM, "the output rows fit the staging memory");
    const float inv = 1.f / p.dscale[bg];
    uint16_t* rows = smem + wave * OUT_ROWS_ELEMS<D>;
    if (qh == 0)
      store_grad_rows<D, ROPE>(dk, p.scale * inv, static_cast<uint16_t*>(p.dk) + (size_t)bg * S * D, p.table, nw, S,
                               rows, lane);
    else
      store_grad_rows<D, ROPE_NONE>(dv, inv, static_cast<uint16_t*>(p.dv) + (size_t)bg * S * D, nullptr, nw, S, rows,
                                    lane);
  }
}

// Convert a staged K tile's registers from bf16 to fp16 (exact for |k| < 65504).
template <int D>
__device__ __forceinline__ void k_to_f16(TileRegs<D, ROPE_NONE>& R) {
  using C = TileCfg<D, ROPE_NONE>;
#pragma unroll
  for (int i = 0; i < C::KPT; ++i)
#pragma unroll
    for (int w = 0; w < 4; ++w) R.ka[i][w] = pack_f16(bf_lo(R.ka[i][w]), bf_hi(R.ka[i][w]));
}

// ---------------------------------------------------------------- dQ
// LDS layout of the dQ pass's key tiles: K' is read by rows (S^T = K' Q'^T)
// and transposed (dQ'^T += K'^T dS^T), so it is stored swizzled (swz_at, no
// padding); V is read by rows only, at a pitch of D + 8 (16-byte reads of 16
// rows fall in distinct banks).
template <int D>
struct DqTileCfg {
  static constexpr int K_ELEMS = 64 * D;
  static constexpr int VP = D + 8;
  static constexpr int STAGE = K_ELEMS + 64 * VP;
};

// Commit a staged key tile (tile_load layout of TileCfg<D, ROPE_NONE>) into
// the dQ pass's layout.
template <int D>
__device__ __forceinline__ void dq_tile_commit(const TileRegs<D, ROPE_NONE>& R, uint16_t* __restrict__ Ks,
                                               uint16_t* __restrict__ Vs, int tid) {
  using C = TileCfg<D, ROPE_NONE>;
#pragma unroll
  for (int i = 0; i < C::KPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::K_ITEMS % C::THREADS != 0 && it >= C::K_ITEMS) break;
    const int r = it / C::K_UNITS, c = it % C::K_UNITS;
    *reinterpret_cast<u32x4*>(Ks + swz_at<D>(r, 8 * c)) = R.ka[i];
  }
#pragma unroll
  for (int i = 0; i < C::VPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::V_ITEMS % C::THREADS != 0 && it >= C::V_ITEMS) break;
    const int r = it / (D / 8), c = it % (D / 8);
    *reinterpret_cast<u32x4*>(Vs + r * DqTileCfg<D>::VP + 8 * c) = R.v[i];
  }
}

// Same decomposition as the forward: 8 waves, GQA heads packed, double-buffered
// K'/V tiles (loaded as attn_tiles.hpp does, stored in the layout above);
// dQ'^T += K'^T dS^T with K'^T from transpose reads.
template <int D, int ROPE, int MASK, bool ALIBI, bool SPARSE, int EXT = EXT_NONE>
__global__ __launch_bounds__(512) void bwd_dq_kernel(BwdParams p) {
  using C = TileCfg<D, ROPE_NONE>;            // K' arrives rotated, or K is converted to fp16 at staging
  using L = DqTileCfg<D>;
  constexpr bool ROT = ROPE != ROPE_NONE;    // Q' and K' come rotated (fp16) from the workspace
  constexpr bool TBIAS = EXT == EXT_BIAS || EXT == EXT_RELU_BIAS;
  constexpr bool RELU = EXT == EXT_RELU || EXT == EXT_RELU_BIAS;
  static_assert(TILE_LIST_SCRATCH_BYTES <= 2 * L::STAGE * (int)sizeof(uint16_t), "the tile-list scratch fits the stages");
  // the two key-tile stages, and at the end each wave's dQ rows on their way out
  constexpr int SMEM = (2 * L::STAGE > C::NW * OUT_ROWS_ELEMS<D>) ? 2 * L::STAGE : C::NW * OUT_ROWS_ELEMS<D>;
  __shared__ __attribute__((aligned(16))) uint16_t smem[SMEM];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, lq = lane & 31, lg = lane >> 5;
  const int S = p.S;
  const int HP = p.heads_per_wg;
  const int WPH = C::NW / HP;
  const int P = 32 * WPH;
  const int G = p.H / p.Hkv;
  const int groups = G / HP;
  const int units = p.B * p.Hkv * groups;
  const int npb = (S + P - 1) / P;
  const int unit = blockIdx.x % units;
  // position blocks run backwards (the longest causal rows first); under a
  // block mask without an elementwise mask they run forwards, as the forward's
  // do, which starts global rows (conventionally the first) early
  const int pb = (SPARSE && MASK == MASK_NONE) ? (int)(blockIdx.x / units) : npb - 1 - (int)(blockIdx.x / units);
  const int hg = unit % groups, bg = unit / groups;
  const int b = bg / p.Hkv, g = bg % p.Hkv;
  const int h = g * G + hg * HP + wave / WPH;
  const int p0 = pb * P;
  const int mw = p0 + 32 * (wave % WPH);
  const int m = mw + lq;
  const int p_end = min(p0 + P, S);
  const size_t bh = (size_t)b * p.H + h;

  const uint16_t* Qh = static_cast<const uint16_t*>(ROT ? p.qr16 : p.q) + bh * S * D;
  const uint16_t* dOh = static_cast<const uint16_t*>(p.dout) + bh * S * D;
  const uint16_t* Kg = static_cast<const uint16_t*>(ROT ? p.kr16 : p.k) + (size_t)bg * S * D;
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v) + (size_t)bg * S * D;

  u32x4 qreg[C::KS], oreg[C::KS];
  const int mc = min(m, S - 1);   // rows past S compute on row S-1 and are never stored
  load_row_operand<D, ROPE_NONE, !ROT>(qreg, Qh, nullptr, mc, S, lg);
  load_row_operand<D, ROPE_NONE>(oreg, dOh, nullptr, mc, S, lg);
  const float lse2 = (m < S) ? p.lse2[bh * S + mc] : INFINITY;
  const float* __restrict__ brow = nullptr;       // this lane's row of the bias tensor
  if constexpr (TBIAS) brow = p.bias + b * p.bias_sb + h * p.bias_sh + mc * p.bias_sq;
  const float del = (m < S) ? p.delta[bh * S + mc] : 0.f;   // sigma delta_i from rowsum(dO o O)
  const float sig = p.dscale[bg];
  float dsum = 0.f;   // this lane's part of sum_j P_ij dP_ij (unscaled)
  float lsum = 0.f;   // and of sum_j P_ij

  f32x16 dq[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) dq[i] = f32x16{};

  const float c2 = p.scale * kLog2e;
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;
  const int W = p.window;
  const int ntiles = (S + C::BN - 1) / C::BN;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (p_end - 1) / C::BN + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, p0 - W + 1) / C::BN;

  // Key tiles by position i: t_begin + i, or under a block-sparse mask the
  // union of the workgroup's query blocks' active key blocks (as the forward).
  __shared__ std::conditional_t<SPARSE, TileList<true>, int> tl;
  int ntl = t_end - t_begin;
  int jw = 0;
  if constexpr (SPARSE) {             // the staging memory serves as scratch: nothing is staged yet
    const int r0 = p0 / C::BN, r1 = (p_end - 1) / C::BN;
    ntl = __builtin_amdgcn_readfirstlane(build_tile_list<C::THREADS>(tl, smem, p.bq_ptr, p.bk_idx, r0, r1 - r0 + 1,
                                                                     ntiles, t_begin, t_end, tid));
    jw = mw / C::BN - r0;
  }
  auto tile_at = [&](int i) -> int {
    if constexpr (SPARSE) return __builtin_amdgcn_readfirstlane((int)tl.tile[i]);
    else return t_begin + i;
  };

  const SwzLane<D> zl(lane);
  TileRegs<D, ROPE_NONE> R;
  if (ntl > 0) {
    tile_load<D, ROPE_NONE>(R, Kg, Vg, nullptr, tile_at(0) * C::BN, S, tid);
    if constexpr (!ROT) k_to_f16(R);
    dq_tile_commit<D>(R, smem, smem + L::K_ELEMS, tid);
  }
  __syncthreads();

  for (int t = 0; t < ntl; ++t) {
    const int n0 = tile_at(t) * C::BN;
    const SwzLane<D> z = zl.opaque();
    const uint16_t* Ks = smem + (t & 1) * L::STAGE;
    const uint16_t* Vs = Ks + L::K_ELEMS;
    const bool more = t + 1 < ntl;
    if (more) tile_load<D, ROPE_NONE>(R, Kg, Vg, nullptr, tile_at(t + 1) * C::BN, S, tid);

    bool visible = mw < S;
    if constexpr (SPARSE) visible = visible && ((tl.rows[t] >> jw) & 1);
    if constexpr (MASK != MASK_NONE) visible = visible && (n0 <= mw + 31);
    if constexpr (MASK == MASK_SLIDING_WINDOW) visible = visible && (n0 + C::BN - 1 > mw - W);
    if (visible) {
      bool need_mask = n0 + C::BN > S;
      if constexpr (MASK != MASK_NONE) need_mask = need_mask || (n0 + C::BN - 1 > mw);
      if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (n0 <= mw + 31 - W);
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        f32x16 sc = f32x16{}, dp = f32x16{};
#pragma unroll
        for (int k = 0; k < C::KS; ++k) {
          const u32x4 ak = row_operand_swz<D>(Ks, z, 32 * kt, k);
          const u32x4 av = *reinterpret_cast<const u32x4*>(Vs + (32 * kt + lq) * L::VP + 16 * k + 8 * lg);
          sc = mfma32<true>(ak, qreg[k], sc);
          dp = mfma32(av, oreg[k], dp);
        }
        // element r: key nn = n0 + 32 kt + 8 (r/4) + 4 lg + r%4, query m
        float ds[16];
        bool pos[16];   // relu attention: s > 0
        float bias[16] = {};
        if constexpr (TBIAS) load_bias16(bias, brow, n0 + 32 * kt, lg, S);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int nn = n0 + 32 * kt + 8 * (r >> 2) + 4 * lg + (r & 3);
          if constexpr (TBIAS || RELU) {
            const float bv = bias[r];
            if constexpr (RELU) {
              pos[r] = __builtin_fmaf(sc[r], p.scale, bv) > 0.f;
              ds[r] = 1.f;
            } else {
              ds[r] = fast_exp2(__builtin_fmaf(sc[r], c2, bv * kLog2e) - lse2);
            }
          } else {
            const float x = ALIBI ? __builtin_fmaf(sc[r], c2, slope2 * (float)(nn - m)) : sc[r] * c2;
            ds[r] = fast_exp2(x - lse2);
          }
        }
        if (need_mask) {   // wave-uniform
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int nn = n0 + 32 * kt + 8 * (r >> 2) + 4 * lg + (r & 3);
            bool ok = nn < S;
            if constexpr (MASK != MASK_NONE) ok = ok && (nn <= m);
            if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (nn > m - W);
            ds[r] = ok ? ds[r] : 0.f;
          }
        }
        if constexpr (RELU) {   // dS = dP where s > 0
#pragma unroll
          for (int r = 0; r < 16; ++r) ds[r] = pos[r] ? ds[r] * dp[r] * sig : 0.f;
        } else {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            lsum += ds[r];
            dsum = __builtin_fmaf(ds[r], dp[r], dsum);
            ds[r] *= __builtin_fmaf(dp[r], sig, -del);
          }
        }
        u32x4 db[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int w = 0; w < 4; ++w) db[hf][w] = pack_f16(ds[8 * hf + 2 * w], ds[8 * hf + 2 * w + 1]);
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
          for (int hf = 0; hf < 2; ++hf)
            dq[mt] = mfma32<true>(tr_operand_swz<D>(Ks, z, 32 * kt + 16 * hf, mt), db[hf], dq[mt]);
      }
    }
    if (more) {
      uint16_t* Kn = smem + ((t + 1) & 1) * L::STAGE;
      if constexpr (!ROT) k_to_f16(R);
      dq_tile_commit<D>(R, Kn, Kn + L::K_ELEMS, tid);
    }
    __syncthreads();
  }
  // For the dK/dV pass: the row's probabilities as this pass formed them sum
  // to l = sum_j P_ij, which differs from 1 by the rounding of the LSE it was
  // given (noticeable when scores are large); LSE + log2 l renormalises them,
  // and delta = sum_j P_ij dP_ij / l is the softmax backward's row term of
  // the renormalised P.  Rows with no visible key keep LSE = +inf.
  if constexpr (!RELU) {
    const float ltot = pair_sum(lsum), dtot = pair_sum(dsum);   // the lane pair (l, l ^ 32) holds row m's keys
    if (m < S && lg == 0) {
      const bool any = ltot > 0.f;
      p.delta[bh * S + m] = any ? dtot / ltot * sig : 0.f;
      p.lse2[bh * S + m] = any ? lse2 + __log2f(ltot) : INFINITY;
    }
  }
  // the key loop ended on a barrier after every wave's last LDS read
  store_grad_rows<D, ROPE>(dq, p.scale / sig, static_cast<uint16_t*>(p.dq) + bh * S * D, p.table, mw, S,
                           smem + wave * OUT_ROWS_ELEMS<D>, lane);
}

// ---------------------------------------------------------------- launch
template <int D, int ROPE, int MASK, bool ALIBI, int EXT = EXT_NONE>
static int launch_one(const BwdParams& p, hipStream_t st) {
  constexpr int RPB = 256 / (D / 16);
  const long long qrows = (long long)p.B * p.H * p.S;
  const long long krows = (ROPE != ROPE_NONE) ? (long long)p.B * p.Hkv * p.S : 0;
  const int q_blocks = (int)((qrows + RPB - 1) / RPB);
  const int k_blocks = (int)((krows + RPB - 1) / RPB);
  const unsigned groups = (unsigned)(p.B * p.Hkv);
  hipLaunchKernelGGL((bwd_dmax_kernel<D>), dim3(groups * (unsigned)p.dmax_chunks), dim3(256), 0, st, p);
  hipLaunchKernelGGL(bwd_dscale_kernel, dim3(groups), dim3(256), 0, st, p);
  hipLaunchKernelGGL((bwd_prep_kernel<D, ROPE>), dim3((unsigned)(q_blocks + k_blocks)), dim3(256), 0, st, p, q_blocks);
  using TC = TileCfg<D, ROPE_NONE>;
  BwdParams pq = p;
  pq.heads_per_wg = heads_per_wg(p.H / p.Hkv);
  const int P = TC::ROWS / pq.heads_per_wg;
  const long long qblocks = (long long)((p.S + P - 1) / P) * p.B * p.Hkv * ((p.H / p.Hkv) / pq.heads_per_wg);
  if (EXT == EXT_NONE && p.bq_ptr)
    hipLaunchKernelGGL((bwd_dq_kernel<D, ROPE, MASK, ALIBI, true>), dim3((unsigned)qblocks), dim3(TC::THREADS), 0, st,
                       pq);
  else
    hipLaunchKernelGGL((bwd_dq_kernel<D, ROPE, MASK, ALIBI, false, EXT>), dim3((unsigned)qblocks), dim3(TC::THREADS),
                       0, st, pq);
  // after the dQ pass, which replaced delta by sum_j P_ij dP_ij
  using QC = QTileCfg<D>;
  const int nkb = (p.S + QC::KEYS - 1) / QC::KEYS;
  if (EXT == EXT_NONE && p.bk_ptr)
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, ROPE, MASK, ALIBI, true>), dim3((unsigned)(nkb * p.B * p.Hkv)),
                       dim3(QC::THREADS), 0, st, p);
  else
    hipLaunchKernelGGL((bwd_dkdv_kernel<D, ROPE, MASK, ALIBI, false, EXT>), dim3((unsigned)(nkb * p.B * p.Hkv)),
                       dim3(QC::THREADS), 0, st, p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <int D, int ROPE, int MASK>
static int dispatch_ext(bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  switch (ext) {
    case EXT_NONE: return alibi ? launch_one<D, ROPE, MASK, true>(p, st) : launch_one<D, ROPE, MASK, false>(p, st);
    case EXT_BIAS: return launch_one<D, ROPE, MASK, false, EXT_BIAS>(p, st);
    case EXT_RELU: return launch_one<D, ROPE, MASK, false, EXT_RELU>(p, st);
    case EXT_RELU_BIAS: return launch_one<D, ROPE, MASK, false, EXT_RELU_BIAS>(p, st);
  }
  return -2;
}

template <int D, int ROPE>
static int dispatch_mask(int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  switch (mask) {
    case MASK_NONE: return dispatch_ext<D, ROPE, MASK_NONE>(alibi, ext, p, st);
    case MASK_CAUSAL: return dispatch_ext<D, ROPE, MASK_CAUSAL>(alibi, ext, p, st);
    case MASK_SLIDING_WINDOW: return dispatch_ext<D, ROPE, MASK_SLIDING_WINDOW>(alibi, ext, p, st);
  }
  return -2;
}

template <int D>
static int dispatch_rope(int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return dispatch_mask<D, ROPE_NONE>(mask, alibi, ext, p, st);
    case ROPE_NEOX: return dispatch_mask<D, ROPE_NEOX>(mask, alibi, ext, p, st);
    case ROPE_INTERLEAVED: return dispatch_mask<D, ROPE_INTERLEAVED>(mask, alibi, ext, p, st);
  }
  return -2;
}

int launch_bwd_bf16(int D, int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  if (ext != EXT_NONE && (alibi || p.bq_ptr || p.bk_ptr)) return -2;   // not instantiated
  if (D == 64) return dispatch_rope<64>(rope, mask, alibi, ext, p, st);
  if (D == 128) return dispatch_rope<128>(rope, mask, alibi, ext, p, st);
  return -2;
}

}  // namespace af
