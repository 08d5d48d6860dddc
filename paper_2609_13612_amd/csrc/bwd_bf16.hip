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
//   3. bwd_dkdv:  (bwd_dkdv.hip) one workgroup per 128 keys of one (batch,
//                 K/V head); it loops over the query heads of the GQA group
//                 and their visible query tiles, re-deriving P = exp(S - LSE)
//                 tile by tile:  dV += P^T dO,  dS = P o (dO V^T - delta),
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

#include "bwd_common.hpp"

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
namespace {
struct BwdPasses {
  template <int D, int ROPE, int MASK, bool ALIBI, int EXT>
  static int run(const BwdParams& p, hipStream_t st) {
    constexpr int RPB = 256 / (D / 16);
    const long long qrows = (long long)p.B * p.H * p.S;
    const long long krows = (ROPE != ROPE_NONE) ? (long long)p.B * p.Hkv * p.S : 0;
    const int q_blocks = (int)((qrows + RPB - 1) / RPB);
    const int k_blocks = (int)((krows + RPB - 1) / RPB);
    const unsigned groups = (unsigned)(p.B * p.Hkv);
    hipLaunchKernelGGL((bwd_dmax_kernel<D>), dim3(groups * (unsigned)p.dmax_chunks), dim3(256), 0, st, p);
    hipLaunchKernelGGL(bwd_dscale_kernel, dim3(groups), dim3(256), 0, st, p);
    hipLaunchKernelGGL((bwd_prep_kernel<D, ROPE>), dim3((unsigned)(q_blocks + k_blocks)), dim3(256), 0, st, p,
                       q_blocks);
    using TC = TileCfg<D, ROPE_NONE>;
    BwdParams pq = p;
    pq.heads_per_wg = heads_per_wg(p.H / p.Hkv);
    const int P = TC::ROWS / pq.heads_per_wg;
    const long long qblocks = (long long)((p.S + P - 1) / P) * p.B * p.Hkv * ((p.H / p.Hkv) / pq.heads_per_wg);
    if (EXT == EXT_NONE && p.bq_ptr)
      hipLaunchKernelGGL((bwd_dq_kernel<D, ROPE, MASK, ALIBI, true>), dim3((unsigned)qblocks), dim3(TC::THREADS), 0,
                         st, pq);
    else
      hipLaunchKernelGGL((bwd_dq_kernel<D, ROPE, MASK, ALIBI, false, EXT>), dim3((unsigned)qblocks),
                         dim3(TC::THREADS), 0, st, pq);
    if (hipGetLastError() != hipSuccess) return -3;
    // after the dQ pass, which replaced delta by sum_j P_ij dP_ij
    return launch_bwd_dkdv_bf16(D, ROPE, MASK, ALIBI, EXT, p, st);
  }
};
}  // namespace

int launch_bwd_bf16(int D, int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  return bwd_dispatch<BwdPasses>(D, rope, mask, alibi, ext, p, st);
}

}  // namespace af
