// Fused RoPE + masked attention backward, bf16 MFMA with fp32 accumulation,
// for gfx950.
//
// Three kernels, no atomics (Section 4.4): every output tile has exactly one
// writer.
//   1. bwd_rowstat:  delta_i = rowsum(dO_i * O_i) and LSE_i in log2 units.
//   2. bwd_dkdv:     one workgroup per 128 keys of one (batch, K/V head); it
//                    loops over the query heads of the GQA group and their
//                    visible query tiles, re-deriving P = exp(S - LSE) tile by
//                    tile:  dV += P^T dO,  dS = P o (dO V^T - delta),
//                    dK' += scale dS^T Q'.  K' = R K is rotated once; each Q'
//                    tile is rotated as it is staged.  dK = R^T dK'.
//   3. bwd_dq:       one workgroup per 128 queries of one (batch, head); it
//                    loops over visible key tiles:  dQ' += scale dS K',
//                    dQ = R^T dQ'.
// Register layouts follow the forward: the operand held in registers is the
// MFMA B operand (lane = its row), tiles staged in LDS are the A operand, and
// contractions over queries/keys read a transposed LDS copy stored with the
// perm16 row order that matches the score tile's register order.
//
// Precision follows the forward: with RoPE the rotated Q' and K' (and dS,
// which multiplies them) are fp16 MFMA operands, so P is re-derived from the
// same rounded operands that produced the forward's LSE; without RoPE every
// MFMA operand is bf16.  dV = P^T dO sums P over many queries without
// normalisation, so it runs on fp16 operands (P and dO, the latter converted
// exactly from bf16 when its transposed copy is staged); this bounds the
// accumulated rounding of P at 2^-12 per term and needs |dO| < 65504.
// dP = dO V^T uses the bf16 inputs as they are.
#include "common.hpp"
#include "launch.hpp"

namespace af {

// ---------------------------------------------------------------- row statistics
template <int D>
__global__ __launch_bounds__(256) void bwd_rowstat_kernel(BwdParams p) {
  constexpr int TPR = D / 8;             // threads per row (16 bytes each)
  constexpr int RPB = 256 / TPR;         // rows per block
  const long long rows = (long long)p.B * p.H * p.S;
  const long long row = (long long)blockIdx.x * RPB + threadIdx.x / TPR;
  const int c = threadIdx.x % TPR;
  float acc = 0.f;
  if (row < rows) {
    u32x4 a = ld16(static_cast<const uint16_t*>(p.dout) + row * D + 8 * c);
    u32x4 o = ld16(static_cast<const uint16_t*>(p.o) + row * D + 8 * c);
#pragma unroll
    for (int w = 0; w < 4; ++w) acc += bf_lo(a[w]) * bf_lo(o[w]) + bf_hi(a[w]) * bf_hi(o[w]);
  }
#pragma unroll
  for (int off = TPR / 2; off > 0; off >>= 1) acc += __shfl_xor(acc, off, TPR);
  if (row < rows && c == 0) {
    p.delta[row] = acc;
    const float l = p.lse[row];
    p.lse2[row] = (l == -INFINITY) ? INFINITY : l * kLog2e;
  }
}

// ---------------------------------------------------------------- staging
// Stage rows r0..r0+ROWS-1 of a [S][D] bf16 matrix into LDS as rows [ROWS][RP]
// and, if T_PITCH > 0, transposed as [D][T_PITCH] with row order perm16.
// Rows are optionally RoPE-rotated (position = row index; rotated values in
// fp16 when F16OUT); rows >= S are 0.  T_F16 converts an unrotated bf16
// matrix to fp16 in the transposed copy only.
// Each thread handles 4 consecutive rows x one chunk unit (NeoX: the chunk
// pair c, c + D/2; otherwise one 8-element chunk).
template <int D, int ROPE, int ROWS, int RP, int T_PITCH, bool F16OUT = (ROPE != ROPE_NONE), bool T_F16 = false>
__device__ __forceinline__ void stage_rows(uint16_t* __restrict__ dst, uint16_t* __restrict__ dst_t,
                                           const uint16_t* __restrict__ src,
                                           const float2* __restrict__ table, int r0, int S, int tid) {
  constexpr int UNITS = (ROPE == ROPE_NEOX) ? D / 16 : D / 8;
  constexpr int N = (ROWS / 4) * UNITS;
#pragma unroll
  for (int i = 0; i < (N + 255) / 256; ++i) {
    const int it = tid + 256 * i;
    if (N % 256 != 0 && it >= N) break;
    const int j = it / UNITS, u = it % UNITS;
    constexpr int NCH = (ROPE == ROPE_NEOX) ? 2 : 1;
    const int d0[2] = {8 * u, 8 * u + D / 2};
    u32x4 v[4][NCH];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int n = r0 + 4 * j + b;
#pragma unroll
      for (int k = 0; k < NCH; ++k) v[b][k] = u32x4{0, 0, 0, 0};
      if (n < S) {
#pragma unroll
        for (int k = 0; k < NCH; ++k) v[b][k] = ld16(src + (size_t)n * D + d0[k]);
        if constexpr (ROPE == ROPE_NEOX)
          rotate_neox8<false, F16OUT>(v[b][0], v[b][1], table + (size_t)n * (D / 2) + 8 * u);
        if constexpr (ROPE == ROPE_INTERLEAVED)
          rotate_interleaved8<false, F16OUT>(v[b][0], table + (size_t)n * (D / 2) + 4 * u);
      }
#pragma unroll
      for (int k = 0; k < NCH; ++k) *reinterpret_cast<u32x4*>(dst + (4 * j + b) * RP + d0[k]) = v[b][k];
    }
    if constexpr (T_PITCH > 0) {
      static_assert(!(T_F16 && ROPE != ROPE_NONE), "T_F16 converts unrotated bf16 rows only");
      if constexpr (T_F16) {
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int k = 0; k < NCH; ++k)
#pragma unroll
            for (int w = 0; w < 4; ++w) v[b][k][w] = pack_f16(bf_lo(v[b][k][w]), bf_hi(v[b][k][w]));
      }
      const int col = perm16(4 * j);
#pragma unroll
      for (int k = 0; k < NCH; ++k) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          u32x2 lo = {(v[0][k][w] & 0xffffu) | (v[1][k][w] << 16), (v[2][k][w] & 0xffffu) | (v[3][k][w] << 16)};
          u32x2 hi = {(v[0][k][w] >> 16) | (v[1][k][w] & 0xffff0000u), (v[2][k][w] >> 16) | (v[3][k][w] & 0xffff0000u)};
          *reinterpret_cast<u32x2*>(dst_t + (d0[k] + 2 * w) * T_PITCH + col) = lo;
          *reinterpret_cast<u32x2*>(dst_t + (d0[k] + 2 * w + 1) * T_PITCH + col) = hi;
        }
      }
    }
  }
}

// Load one lane's row of a bf16 matrix as the MFMA B operand (dims 16s + 8lg..+7),
// RoPE-rotated in-lane (rotated values rounded to fp16).  Rows >= S give zeros.
template <int D, int ROPE>
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
}

// Scale, undo the rotation and store an accumulator tile X^T (d x rows) whose
// lane owns row n: element r of tile mt is dim 32 mt + 8 (r/4) + 4 lg + r%4.
template <int D, int ROPE>
__device__ __forceinline__ void store_grad_rows(f32x16 (&acc)[D / 32], float scale, uint16_t* __restrict__ dst,
                                                const float2* __restrict__ table, int n, int lg) {
  constexpr int MT = D / 32;
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
  uint16_t* row = dst + (size_t)n * D;
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      u32x2 w = {pack_bf16(acc[mt][4 * a], acc[mt][4 * a + 1]), pack_bf16(acc[mt][4 * a + 2], acc[mt][4 * a + 3])};
      *reinterpret_cast<u32x2*>(row + 32 * mt + 8 * a + 4 * lg) = w;
    }
  }
}

template <int D>
struct BwdCfg {
  static constexpr int BQ = 64;         // query rows per staged tile (dK/dV kernel)
  static constexpr int BK = 64;         // key rows per staged tile (dQ kernel)
  static constexpr int KS = D / 16;
  static constexpr int MT = D / 32;
  static constexpr int RP = D + 8;      // LDS pitch of [rows][D] tiles
  static constexpr int TP = 64 + 8;     // LDS pitch of [D][64] transposed tiles
};

// ---------------------------------------------------------------- dK / dV
template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(256) void bwd_dkdv_kernel(BwdParams p) {
  using C = BwdCfg<D>;
  constexpr bool QF16 = ROPE != ROPE_NONE;   // rotated operands (and dS with them) in fp16
  __shared__ __attribute__((aligned(16))) uint16_t Qs[C::BQ * C::RP];
  __shared__ __attribute__((aligned(16))) uint16_t Qt[D * C::TP];
  __shared__ __attribute__((aligned(16))) uint16_t Os[C::BQ * C::RP];   // dO rows
  __shared__ __attribute__((aligned(16))) uint16_t Ot[D * C::TP];       // dO^T, fp16
  __shared__ __attribute__((aligned(16))) float lse2s[C::BQ];
  __shared__ __attribute__((aligned(16))) float dels[C::BQ];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, lq = lane & 31, lg = lane >> 5;
  const int S = p.S;
  const int nkb = (S + 127) / 128;
  const int BG = p.B * p.Hkv;
  const int bg = blockIdx.x % BG;
  const int kb = nkb - 1 - (int)(blockIdx.x / BG);
  const int b = bg / p.Hkv, g = bg % p.Hkv;
  const int G = p.H / p.Hkv;
  const int nb = kb * 128;            // first key of the block
  const int nw = nb + 32 * wave;      // first key of this wave
  const int n = nw + lq;              // this lane's key

  const uint16_t* Kg = static_cast<const uint16_t*>(p.k) + (size_t)bg * S * D;
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v) + (size_t)bg * S * D;
  u32x4 kreg[C::KS], vreg[C::KS];
  load_row_operand<D, ROPE>(kreg, Kg, p.table, n, S, lg);
  load_row_operand<D, ROPE_NONE>(vreg, Vg, nullptr, n, S, lg);

  f32x16 dk[C::MT], dv[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) { dk[i] = f32x16{}; dv[i] = f32x16{}; }

  const float c2 = p.scale * kLog2e;
  const int W = p.window;
  const int ntq = (S + C::BQ - 1) / C::BQ;
  int tq_begin = 0, tq_end = ntq;
  if constexpr (MASK != MASK_NONE) tq_begin = nb / C::BQ;
  if constexpr (MASK == MASK_SLIDING_WINDOW) tq_end = min(ntq, (min(nb + 127, S - 1) + W - 1) / C::BQ + 1);

  for (int hq = 0; hq < G; ++hq) {
    const int h = g * G + hq;
    const size_t bh = (size_t)b * p.H + h;
    const uint16_t* Qh = static_cast<const uint16_t*>(p.q) + bh * S * D;
    const uint16_t* dOh = static_cast<const uint16_t*>(p.dout) + bh * S * D;
    const float* lse2h = p.lse2 + bh * S;
    const float* delh = p.delta + bh * S;
    const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;

    for (int tq = tq_begin; tq < tq_end; ++tq) {
      const int mq0 = tq * C::BQ;
      __syncthreads();
      stage_rows<D, ROPE, C::BQ, C::RP, C::TP>(Qs, Qt, Qh, p.table, mq0, S, tid);
      stage_rows<D, ROPE_NONE, C::BQ, C::RP, C::TP, false, true>(Os, Ot, dOh, nullptr, mq0, S, tid);
      if (tid < C::BQ) {
        const int m = mq0 + tid;
        lse2s[tid] = (m < S) ? lse2h[m] : INFINITY;
        dels[tid] = (m < S) ? delh[m] : 0.f;
      }
      __syncthreads();

      bool visible = nw < S;
      if constexpr (MASK != MASK_NONE) visible = visible && (mq0 + C::BQ - 1 >= nw);
      if constexpr (MASK == MASK_SLIDING_WINDOW) visible = visible && (mq0 <= nw + 31 + W - 1);
      if (!visible) continue;
      bool need_mask = nw + 32 > S;
      if constexpr (MASK != MASK_NONE) need_mask = need_mask || (mq0 < nw + 31);
      if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (mq0 + C::BQ - 1 - W >= nw);

#pragma unroll
      for (int qt = 0; qt < 2; ++qt) {
        f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
        for (int k = 0; k < C::KS; ++k) {
          u32x4 aq = *reinterpret_cast<const u32x4*>(Qs + (32 * qt + lq) * C::RP + 16 * k + 8 * lg);
          s = mfma32<QF16>(aq, kreg[k], s);
        }
#pragma unroll
        for (int k = 0; k < C::KS; ++k) {
          u32x4 ao = *reinterpret_cast<const u32x4*>(Os + (32 * qt + lq) * C::RP + 16 * k + 8 * lg);
          dp = mfma32(ao, vreg[k], dp);
        }
        // element r: query ql = 32 qt + 8 (r/4) + 4 lg + r%4, key n
        float pr[16], ds[16];
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
            const int m = mq0 + qlb + e;
            float x = ALIBI ? __builtin_fmaf(s[r], c2, slope2 * (float)(n - m)) : s[r] * c2;
            float pv = fast_exp2(x - lv[e]);
            if (need_mask) {
              bool ok = n < S;
              if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
              if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
              if (!ok) pv = 0.f;
            }
            pr[r] = pv;
            ds[r] = pv * (dp[r] - dv4[e]);
          }
        }
        u32x4 pb[2], db[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            pb[hf][w] = pack_f16(pr[8 * hf + 2 * w], pr[8 * hf + 2 * w + 1]);
            db[hf][w] = pack_op<QF16>(ds[8 * hf + 2 * w], ds[8 * hf + 2 * w + 1]);
          }
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
#pragma unroll
          for (int hf = 0; hf < 2; ++hf) {
            const int col = 32 * qt + 16 * hf + 8 * lg;
            u32x4 ao = *reinterpret_cast<const u32x4*>(Ot + (32 * mt + lq) * C::TP + col);
            dv[mt] = mfma32<true>(ao, pb[hf], dv[mt]);
            u32x4 aq = *reinterpret_cast<const u32x4*>(Qt + (32 * mt + lq) * C::TP + col);
            dk[mt] = mfma32<QF16>(aq, db[hf], dk[mt]);
          }
        }
      }
    }
  }

  if (n < S) {
    store_grad_rows<D, ROPE>(dk, p.scale, static_cast<uint16_t*>(p.dk) + (size_t)bg * S * D, p.table, n, lg);
    store_grad_rows<D, ROPE_NONE>(dv, 1.f, static_cast<uint16_t*>(p.dv) + (size_t)bg * S * D, nullptr, n, lg);
  }
}

// ---------------------------------------------------------------- dQ
template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(256) void bwd_dq_kernel(BwdParams p) {
  using C = BwdCfg<D>;
  constexpr bool QF16 = ROPE != ROPE_NONE;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[C::BK * C::RP];
  __shared__ __attribute__((aligned(16))) uint16_t Kt[D * C::TP];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[C::BK * C::RP];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, lq = lane & 31, lg = lane >> 5;
  const int S = p.S;
  const int BH = p.B * p.H;
  const int nqb = (S + 127) / 128;
  const int bh = blockIdx.x % BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / BH);
  const int b = bh / p.H, h = bh % p.H;
  const int g = h / (p.H / p.Hkv);
  const int m0 = qb * 128;
  const int mw = m0 + 32 * wave;
  const int m = mw + lq;

  const uint16_t* Qh = static_cast<const uint16_t*>(p.q) + (size_t)bh * S * D;
  const uint16_t* dOh = static_cast<const uint16_t*>(p.dout) + (size_t)bh * S * D;
  const uint16_t* Kg = static_cast<const uint16_t*>(p.k) + (size_t)(b * p.Hkv + g) * S * D;
  const uint16_t* Vg = static_cast<const uint16_t*>(p.v) + (size_t)(b * p.Hkv + g) * S * D;

  u32x4 qreg[C::KS], oreg[C::KS];
  load_row_operand<D, ROPE>(qreg, Qh, p.table, m, S, lg);
  load_row_operand<D, ROPE_NONE>(oreg, dOh, nullptr, m, S, lg);
  const float lse2 = (m < S) ? p.lse2[(size_t)bh * S + m] : INFINITY;
  const float del = (m < S) ? p.delta[(size_t)bh * S + m] : 0.f;

  f32x16 dq[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) dq[i] = f32x16{};

  const float c2 = p.scale * kLog2e;
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;
  const int W = p.window;
  const int ntiles = (S + C::BK - 1) / C::BK;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (min(m0 + 128, S) - 1) / C::BK + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, m0 - W + 1) / C::BK;

  for (int t = t_begin; t < t_end; ++t) {
    const int n0 = t * C::BK;
    __syncthreads();
    stage_rows<D, ROPE, C::BK, C::RP, C::TP>(Ks, Kt, Kg, p.table, n0, S, tid);
    stage_rows<D, ROPE_NONE, C::BK, C::RP, 0>(Vs, nullptr, Vg, nullptr, n0, S, tid);
    __syncthreads();

    bool visible = mw < S;
    if constexpr (MASK != MASK_NONE) visible = visible && (n0 <= mw + 31);
    if constexpr (MASK == MASK_SLIDING_WINDOW) visible = visible && (n0 + C::BK - 1 > mw - W);
    if (!visible) continue;
    bool need_mask = n0 + C::BK > S;
    if constexpr (MASK != MASK_NONE) need_mask = need_mask || (n0 + C::BK - 1 > mw);
    if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (n0 <= mw + 31 - W);

#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      f32x16 s = f32x16{}, dp = f32x16{};
#pragma unroll
      for (int k = 0; k < C::KS; ++k) {
        u32x4 ak = *reinterpret_cast<const u32x4*>(Ks + (32 * kt + lq) * C::RP + 16 * k + 8 * lg);
        s = mfma32<QF16>(ak, qreg[k], s);
      }
#pragma unroll
      for (int k = 0; k < C::KS; ++k) {
        u32x4 av = *reinterpret_cast<const u32x4*>(Vs + (32 * kt + lq) * C::RP + 16 * k + 8 * lg);
        dp = mfma32(av, oreg[k], dp);
      }
      // element r: key nn = n0 + 32 kt + 8 (r/4) + 4 lg + r%4, query m
      float ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int nn = n0 + 32 * kt + 8 * (r >> 2) + 4 * lg + (r & 3);
        float x = ALIBI ? __builtin_fmaf(s[r], c2, slope2 * (float)(nn - m)) : s[r] * c2;
        float pv = fast_exp2(x - lse2);
        if (need_mask) {
          bool ok = nn < S;
          if constexpr (MASK != MASK_NONE) ok = ok && (nn <= m);
          if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (nn > m - W);
          if (!ok) pv = 0.f;
        }
        ds[r] = pv * (dp[r] - del);
      }
      u32x4 db[2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int w = 0; w < 4; ++w) db[hf][w] = pack_op<QF16>(ds[8 * hf + 2 * w], ds[8 * hf + 2 * w + 1]);
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          u32x4 ak = *reinterpret_cast<const u32x4*>(Kt + (32 * mt + lq) * C::TP + 32 * kt + 16 * hf + 8 * lg);
          dq[mt] = mfma32<QF16>(ak, db[hf], dq[mt]);
        }
      }
    }
  }
  if (m < S) store_grad_rows<D, ROPE>(dq, p.scale, static_cast<uint16_t*>(p.dq) + (size_t)bh * S * D, p.table, m, lg);
}

// ---------------------------------------------------------------- launch
template <int D, int ROPE, int MASK, bool ALIBI>
static int launch_one(const BwdParams& p, hipStream_t st) {
  constexpr int RPB = 256 / (D / 8);
  const long long rows = (long long)p.B * p.H * p.S;
  hipLaunchKernelGGL(bwd_rowstat_kernel<D>, dim3((unsigned)((rows + RPB - 1) / RPB)), dim3(256), 0, st, p);
  const int nkb = (p.S + 127) / 128;
  hipLaunchKernelGGL((bwd_dkdv_kernel<D, ROPE, MASK, ALIBI>), dim3((unsigned)(nkb * p.B * p.Hkv)), dim3(256), 0, st, p);
  hipLaunchKernelGGL((bwd_dq_kernel<D, ROPE, MASK, ALIBI>), dim3((unsigned)(nkb * p.B * p.H)), dim3(256), 0, st, p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <int D, int ROPE>
static int dispatch_mask(int mask, bool alibi, const BwdParams& p, hipStream_t st) {
  switch (mask) {
    case MASK_NONE: return alibi ? launch_one<D, ROPE, MASK_NONE, true>(p, st) : launch_one<D, ROPE, MASK_NONE, false>(p, st);
    case MASK_CAUSAL: return alibi ? launch_one<D, ROPE, MASK_CAUSAL, true>(p, st) : launch_one<D, ROPE, MASK_CAUSAL, false>(p, st);
    case MASK_SLIDING_WINDOW: return alibi ? launch_one<D, ROPE, MASK_SLIDING_WINDOW, true>(p, st) : launch_one<D, ROPE, MASK_SLIDING_WINDOW, false>(p, st);
  }
  return -2;
}

template <int D>
static int dispatch_rope(int rope, int mask, bool alibi, const BwdParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return dispatch_mask<D, ROPE_NONE>(mask, alibi, p, st);
    case ROPE_NEOX: return dispatch_mask<D, ROPE_NEOX>(mask, alibi, p, st);
    case ROPE_INTERLEAVED: return dispatch_mask<D, ROPE_INTERLEAVED>(mask, alibi, p, st);
  }
  return -2;
}

int launch_bwd_bf16(int D, int rope, int mask, bool alibi, const BwdParams& p, hipStream_t st) {
  if (D == 64) return dispatch_rope<64>(rope, mask, alibi, p, st);
  if (D == 128) return dispatch_rope<128>(rope, mask, alibi, p, st);
  return -2;
}

}  // namespace af
