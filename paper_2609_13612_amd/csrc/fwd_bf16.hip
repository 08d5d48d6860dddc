// Fused RoPE + masked attention forward, bf16 inputs, bf16 MFMA with fp32
// accumulation, for gfx950.
//
// Method (AttnFuse, Section 2 online softmax, Section 4.1 fused RoPE): the
// query block is rotated once before the key loop; every key tile is rotated
// on the fly as it is staged into LDS; the post-matmul modifications (ALiBi,
// causal, sliding window) are applied to the scores in registers; fully
// masked key tiles are never visited.
//
// Work decomposition
//   workgroup = 4 waves = 128 query rows of one (batch, head); wave = 32 rows.
//   Key tiles of BN = 64 rows are staged in LDS and shared by the 4 waves.
//   Scores are formed transposed, S^T = K' Q'^T (keys x queries), so every
//   lane owns ONE query column and 16 keys per 32x32 MFMA tile: the row max
//   is an in-lane reduction plus a single swap with lane l^32, and the row
//   sum stays per lane until the epilogue.  P^T then feeds O^T += V^T P^T
//   straight from registers as the B operand; V is stored transposed in LDS
//   with the bit-2/3 key permutation that lines the keys up with P^T's
//   register order.
//
// Precision: without RoPE the bf16 inputs feed Q K^T exactly.  With RoPE the
// rotated Q' and K' must be rounded to some 16-bit MFMA operand type; they are
// rounded to fp16 (11-bit significand) rather than bf16 (8-bit), which keeps
// the row statistic LSE within 1e-3 of the exact value.  The fp16 range then
// bounds the rotated inputs: |q|, |k| well below 65504.  P and V stay bf16.
#include "common.hpp"
#include "launch.hpp"

namespace af {

template <int D>
struct FwdCfg {
  static constexpr int NW = 4;          // waves per workgroup
  static constexpr int BM = 32 * NW;    // query rows per workgroup
  static constexpr int BN = 64;         // keys per tile
  static constexpr int KS = D / 16;     // MFMA k-steps over the head dimension
  static constexpr int MT = D / 32;     // 32-row output tiles over the head dimension
  static constexpr int KROW = D + 8;    // LDS pitch (bf16) of the K tile   [BN][KROW]
  static constexpr int VROW = BN + 8;   // LDS pitch (bf16) of the V^T tile [D][VROW]
};

// Stage key tile n0..n0+BN-1 into LDS: K rotated (RoPE) as [key][d], V as
// V^T [d][perm16(key)].  Rows at or beyond S are zero.
template <int D, int ROPE>
__device__ __forceinline__ void stage_kv_tile(uint16_t* __restrict__ Ks, uint16_t* __restrict__ Vt,
                                              const uint16_t* __restrict__ K,
                                              const uint16_t* __restrict__ V,
                                              const float2* __restrict__ table, int n0, int S,
                                              int tid) {
  using C = FwdCfg<D>;
  if constexpr (ROPE == ROPE_NEOX) {
    constexpr int CP = D / 16;   // chunk pairs per row: chunk c and chunk c + D/16
    constexpr int N = C::BN * CP;
#pragma unroll
    for (int i = 0; i < (N + 255) / 256; ++i) {
      const int it = tid + 256 * i;
      if (N % 256 != 0 && it >= N) break;
      const int r = it / CP, c = it % CP, n = n0 + r;
      u32x4 a = {0, 0, 0, 0}, b = {0, 0, 0, 0};
      if (n < S) {
        a = ld16(K + (size_t)n * D + 8 * c);
        b = ld16(K + (size_t)n * D + D / 2 + 8 * c);
        rotate_neox8<false, true>(a, b, table + (size_t)n * (D / 2) + 8 * c);
      }
      *reinterpret_cast<u32x4*>(Ks + r * C::KROW + 8 * c) = a;
      *reinterpret_cast<u32x4*>(Ks + r * C::KROW + D / 2 + 8 * c) = b;
    }
  } else {
    constexpr int CH = D / 8;    // 16-byte chunks per row
    constexpr int N = C::BN * CH;
#pragma unroll
    for (int i = 0; i < (N + 255) / 256; ++i) {
      const int it = tid + 256 * i;
      if (N % 256 != 0 && it >= N) break;
      const int r = it / CH, c = it % CH, n = n0 + r;
      u32x4 a = {0, 0, 0, 0};
      if (n < S) {
        a = ld16(K + (size_t)n * D + 8 * c);
        if constexpr (ROPE == ROPE_INTERLEAVED)
          rotate_interleaved8<false, true>(a, table + (size_t)n * (D / 2) + 4 * c);
      }
      *reinterpret_cast<u32x4*>(Ks + r * C::KROW + 8 * c) = a;
    }
  }
  // V^T: each thread transposes a 4-key x 8-dim block.
  constexpr int OCT = D / 8;
  constexpr int NV = (C::BN / 4) * OCT;
#pragma unroll
  for (int i = 0; i < (NV + 255) / 256; ++i) {
    const int it = tid + 256 * i;
    if (NV % 256 != 0 && it >= NV) break;
    const int j = it / OCT, o = it % OCT;
    u32x4 r[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int n = n0 + 4 * j + b;
      r[b] = (n < S) ? ld16(V + (size_t)n * D + 8 * o) : u32x4{0, 0, 0, 0};
    }
    const int col = perm16(4 * j);
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      u32x2 lo = {(r[0][w] & 0xffffu) | (r[1][w] << 16), (r[2][w] & 0xffffu) | (r[3][w] << 16)};
      u32x2 hi = {(r[0][w] >> 16) | (r[1][w] & 0xffff0000u), (r[2][w] >> 16) | (r[3][w] & 0xffff0000u)};
      *reinterpret_cast<u32x2*>(Vt + (8 * o + 2 * w) * C::VROW + col) = lo;
      *reinterpret_cast<u32x2*>(Vt + (8 * o + 2 * w + 1) * C::VROW + col) = hi;
    }
  }
}

template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(256) void fwd_bf16_kernel(FwdParams p) {
  using C = FwdCfg<D>;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[C::BN * C::KROW];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[D * C::VROW];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lq = lane & 31, lg = lane >> 5;
  const int S = p.S;
  const int BH = p.B * p.H;
  const int nqb = (S + C::BM - 1) / C::BM;
  // Longest (last) query blocks first; all blocks of one head share
  // blockIdx % (B*H), so with B*H a multiple of 8 they land on one XCD.
  const int bh = blockIdx.x % BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / BH);
  const int b = bh / p.H, h = bh % p.H;
  const int g = h / (p.H / p.Hkv);
  const int m0 = qb * C::BM;
  const int mw = m0 + wave * 32;
  const int m = mw + lq;

  const uint16_t* __restrict__ Q = static_cast<const uint16_t*>(p.q) + (size_t)bh * S * D;
  const uint16_t* __restrict__ K = static_cast<const uint16_t*>(p.k) + (size_t)(b * p.Hkv + g) * S * D;
  const uint16_t* __restrict__ V = static_cast<const uint16_t*>(p.v) + (size_t)(b * p.Hkv + g) * S * D;

  // Query operand (B of S^T = K Q^T): lane holds row m, dims 16s + 8lg .. +7.
  u32x4 qreg[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s)
    qreg[s] = (m < S) ? ld16(Q + (size_t)m * D + 16 * s + 8 * lg) : u32x4{0, 0, 0, 0};
  if (m < S) {
    if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
      for (int s = 0; s < C::KS / 2; ++s)
        rotate_neox8<false, true>(qreg[s], qreg[s + C::KS / 2], p.table + (size_t)m * (D / 2) + 16 * s + 8 * lg);
    } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
      for (int s = 0; s < C::KS; ++s)
        rotate_interleaved8<false, true>(qreg[s], p.table + (size_t)m * (D / 2) + 8 * s + 4 * lg);
    }
  }

  const float c2 = p.scale * kLog2e;                          // score -> log2 units
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;   // ALiBi slope, log2 units
  const int W = p.window;

  const int ntiles = (S + C::BN - 1) / C::BN;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (min(m0 + C::BM, S) - 1) / C::BN + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, m0 - W + 1) / C::BN;

  f32x16 acc[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) acc[i] = f32x16{};
  float m_run = -INFINITY;   // running max, log2 units
  float l_run = 0.f;         // this lane's partial row sum

  for (int t = t_begin; t < t_end; ++t) {
    const int n0 = t * C::BN;
    __syncthreads();
    stage_kv_tile<D, ROPE>(Ks, Vt, K, V, p.table, n0, S, tid);
    __syncthreads();

    bool visible = mw < S;
    if constexpr (MASK != MASK_NONE) visible = visible && (n0 <= mw + 31);
    if constexpr (MASK == MASK_SLIDING_WINDOW) visible = visible && (n0 + C::BN - 1 > mw - W);
    if (!visible) continue;   // wave-uniform

    // S^T = K' Q'^T: two 32-key subtiles.
    f32x16 st[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      st[kt] = f32x16{};
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
        u32x4 a = *reinterpret_cast<const u32x4*>(Ks + (32 * kt + lq) * C::KROW + 16 * s + 8 * lg);
        st[kt] = mfma32<(ROPE != ROPE_NONE)>(a, qreg[s], st[kt]);
      }
    }

    bool need_mask = n0 + C::BN > S;
    if constexpr (MASK != MASK_NONE) need_mask = need_mask || (n0 + C::BN - 1 > mw);
    if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (n0 <= mw + 31 - W);

    // Scores in log2 units (ALiBi folded in), masked entries at -inf.
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + 32 * kt + 8 * (r >> 2) + 4 * lg + (r & 3);
        float x = st[kt][r];
        if constexpr (ALIBI) x = __builtin_fmaf(x, c2, slope2 * (float)(n - m));
        if (need_mask) {
          bool ok = n < S;
          if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
          if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
          if (!ok) x = -INFINITY;
        }
        st[kt][r] = x;
      }
    }

    float mx = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[kt][r]);
    mx = pair_max(mx);
    if constexpr (!ALIBI) mx *= c2;
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);

    u32x4 pb[2][2];
    float rs = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      float pv[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float arg = ALIBI ? (st[kt][r] - m_use) : __builtin_fmaf(st[kt][r], c2, -m_use);
        pv[r] = fast_exp2(arg);
        rs += pv[r];
      }
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int w = 0; w < 4; ++w) pb[kt][hf][w] = pack_bf16(pv[8 * hf + 2 * w], pv[8 * hf + 2 * w + 1]);
    }
    l_run = l_run * alpha + rs;
    m_run = m_new;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int i = 0; i < C::MT; ++i) acc[i] *= alpha;
    }

    // O^T += V^T P^T.
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          u32x4 a = *reinterpret_cast<const u32x4*>(Vt + (32 * mt + lq) * C::VROW + 32 * kt + 16 * hf + 8 * lg);
          acc[mt] = mfma32(a, pb[kt][hf], acc[mt]);
        }
      }
    }
  }

  // Epilogue: O = acc / l, LSE = (m + log2 l) ln 2.
  const float l_tot = pair_sum(l_run);
  if (m < S) {
    const float inv = (l_tot > 0.f) ? 1.f / l_tot : 0.f;
    uint16_t* O = static_cast<uint16_t*>(p.o) + ((size_t)bh * S + m) * D;
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        u32x2 w = {pack_bf16(acc[mt][4 * a] * inv, acc[mt][4 * a + 1] * inv),
                   pack_bf16(acc[mt][4 * a + 2] * inv, acc[mt][4 * a + 3] * inv)};
        *reinterpret_cast<u32x2*>(O + 32 * mt + 8 * a + 4 * lg) = w;
      }
    }
    if (lg == 0)
      p.lse[(size_t)bh * S + m] = (l_tot > 0.f) ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

template <int D, int ROPE, int MASK, bool ALIBI>
static int launch_one(const FwdParams& p, hipStream_t st) {
  using C = FwdCfg<D>;
  const int nqb = (p.S + C::BM - 1) / C::BM;
  dim3 grid((unsigned)(nqb * p.B * p.H));
  hipLaunchKernelGGL((fwd_bf16_kernel<D, ROPE, MASK, ALIBI>), grid, dim3(256), 0, st, p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <int D, int ROPE>
static int dispatch_mask(int mask, bool alibi, const FwdParams& p, hipStream_t st) {
  switch (mask) {
    case MASK_NONE: return alibi ? launch_one<D, ROPE, MASK_NONE, true>(p, st) : launch_one<D, ROPE, MASK_NONE, false>(p, st);
    case MASK_CAUSAL: return alibi ? launch_one<D, ROPE, MASK_CAUSAL, true>(p, st) : launch_one<D, ROPE, MASK_CAUSAL, false>(p, st);
    case MASK_SLIDING_WINDOW: return alibi ? launch_one<D, ROPE, MASK_SLIDING_WINDOW, true>(p, st) : launch_one<D, ROPE, MASK_SLIDING_WINDOW, false>(p, st);
  }
  return -2;
}

template <int D>
static int dispatch_rope(int rope, int mask, bool alibi, const FwdParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return dispatch_mask<D, ROPE_NONE>(mask, alibi, p, st);
    case ROPE_NEOX: return dispatch_mask<D, ROPE_NEOX>(mask, alibi, p, st);
    case ROPE_INTERLEAVED: return dispatch_mask<D, ROPE_INTERLEAVED>(mask, alibi, p, st);
  }
  return -2;
}

int launch_fwd_bf16(int D, int rope, int mask, bool alibi, const FwdParams& p, hipStream_t st) {
  if (D == 64) return dispatch_rope<64>(rope, mask, alibi, p, st);
  if (D == 128) return dispatch_rope<128>(rope, mask, alibi, p, st);
  return -2;
}

}  // namespace af
