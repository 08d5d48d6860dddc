// Fused RoPE + masked attention forward, bf16 inputs, MFMA with fp32
// accumulation, for gfx950.
//
// Method (AttnFuse, Section 2 online softmax, Section 4.1 fused RoPE): the
// query rows are rotated once before the key loop; every key tile is rotated
// on the fly as it is staged into LDS; the post-matmul modifications (ALiBi,
// causal, sliding window) are applied to the scores in registers; fully
// masked key tiles are never visited.
//
// Work decomposition
//   workgroup = 8 waves (two per SIMD, so one wave's softmax VALU work runs
//   under the other's MFMA work) = 256 query rows.  The rows are HP query
//   heads of one GQA group x 256/HP positions, so one rotated K tile serves
//   every head that reads it.  Key tiles of BN = 64 rows are double-buffered
//   in LDS: the next tile's K, V and cos/sin are loaded into registers before
//   the current tile is computed and committed (rotated) after it, with one
//   barrier per tile.
//   Scores are formed transposed, S^T = K' Q'^T (keys x queries), so every
//   lane owns ONE query column and 16 keys per 32x32 MFMA tile: the row max
//   is an in-lane reduction plus one v_permlane32_swap, and the row sum stays
//   per lane until the epilogue.  P^T feeds O^T += V^T P^T straight from
//   registers as the B operand; V stays row-major in LDS and its transposed
//   A operand comes from ds_read_b64_tr_b16.
//   The running max is only raised when a row's max grows by more than 2^8,
//   so the O accumulator is rarely rescaled (exact: O and l share the scale).
//
// Precision: without RoPE the bf16 inputs feed Q K^T exactly.  With RoPE the
// rotated Q' and K' are rounded to fp16 (11-bit significand) rather than bf16
// (8-bit), which keeps the row statistic LSE within 1e-3 of the exact value;
// the fp16 range then bounds the rotated inputs (|q|, |k| well below 65504).
// P and V stay bf16.
#include "attn_tiles.hpp"
#include "launch.hpp"

namespace af {

template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(512) void fwd_bf16_kernel(FwdParams p) {
  using C = TileCfg<D, ROPE>;
  constexpr bool QF16 = ROPE != ROPE_NONE;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * C::STAGE];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lq = lane & 31, lg = lane >> 5;
  const int S = p.S;
  // Workgroup -> (batch, K/V head, head group, position block).  The position
  // block is the slow index and runs backwards, so the longest causal blocks
  // start first; consecutive workgroups walk (batch, K/V head, head group), and
  // with that count a multiple of 8 every block of one K/V head lands on the
  // same XCD and shares its L2.
  const int HP = p.heads_per_wg;                 // query heads per workgroup
  const int WPH = C::NW / HP;                    // waves per head
  const int P = 32 * WPH;                        // positions per workgroup
  const int G = p.H / p.Hkv;
  const int groups = G / HP;
  const int units = p.B * p.Hkv * groups;
  const int npb = (S + P - 1) / P;
  const int unit = blockIdx.x % units;
  const int pb = npb - 1 - (int)(blockIdx.x / units);
  const int hg = unit % groups, bg = unit / groups;
  const int b = bg / p.Hkv, g = bg % p.Hkv;
  const int h = g * G + hg * HP + wave / WPH;
  const int p0 = pb * P;
  const int mw = p0 + 32 * (wave % WPH);         // first query row of this wave
  const int m = mw + lq;                         // this lane's query row
  const int p_end = min(p0 + P, S);

  const size_t bh = (size_t)b * p.H + h;
  const uint16_t* __restrict__ Q = static_cast<const uint16_t*>(p.q) + bh * S * D;
  const uint16_t* __restrict__ K = static_cast<const uint16_t*>(p.k) + (size_t)bg * S * D;
  const uint16_t* __restrict__ V = static_cast<const uint16_t*>(p.v) + (size_t)bg * S * D;

  // Query operand (B of S^T = K Q^T): lane holds row m, dims 16s + 8lg .. +7.
  // Rows past S load row S-1 (finite data; never stored).
  const int mc = min(m, S - 1);
  u32x4 qreg[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) qreg[s] = ld16(Q + (size_t)mc * D + 16 * s + 8 * lg);
  if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
    for (int s = 0; s < C::KS / 2; ++s)
      rotate_neox8<false, true>(qreg[s], qreg[s + C::KS / 2], p.table + (size_t)mc * (D / 2) + 16 * s + 8 * lg);
  } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      rotate_interleaved8<false, true>(qreg[s], p.table + (size_t)mc * (D / 2) + 8 * s + 4 * lg);
  }

  const float c2 = p.scale * kLog2e;                          // score -> log2 units
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;   // ALiBi slope, log2 units
  const int W = p.window;

  const int ntiles = (S + C::BN - 1) / C::BN;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (p_end - 1) / C::BN + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, p0 - W + 1) / C::BN;

  f32x16 acc[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) acc[i] = f32x16{};
  float m_run = -INFINITY;   // reference max of the row, log2 units
  float l_run = 0.f;         // this lane's partial row sum (relative to m_run)

  // Transpose-read addressing for the V^T operand (see lds_read_tr16): lane i
  // of each 16-lane group reads 4 dims of key (4 lg + i/4) [+8 for the second
  // read]; the group's 16 lanes cover 16 dims starting at 16 * ((lane/16) & 1).
  const int tr_key = 4 * lg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  TileRegs<D, ROPE> R;
  if (t_begin < t_end) {
    tile_load<D, ROPE>(R, K, V, p.table, t_begin * C::BN, S, tid);
    tile_commit<D, ROPE>(R, smem, smem + C::K_ELEMS, tid);
  }
  __syncthreads();

  for (int t = t_begin; t < t_end; ++t) {
    const int n0 = t * C::BN;
    const uint16_t* Ks = smem + ((t - t_begin) & 1) * C::STAGE;
    const uint16_t* Vs = Ks + C::K_ELEMS;
    const bool more = t + 1 < t_end;
    if (more) tile_load<D, ROPE>(R, K, V, p.table, n0 + C::BN, S, tid);

    bool visible = mw < S;
    if constexpr (MASK != MASK_NONE) visible = visible && (n0 <= mw + 31);
    if constexpr (MASK == MASK_SLIDING_WINDOW) visible = visible && (n0 + C::BN - 1 > mw - W);
    if (visible) {   // wave-uniform
      // S^T = K' Q'^T: two 32-key subtiles, their MFMA chains interleaved.
      f32x16 st[2] = {f32x16{}, f32x16{}};
#pragma unroll
      for (int s = 0; s < C::KS; ++s) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
          u32x4 a = *reinterpret_cast<const u32x4*>(Ks + (32 * kt + lq) * C::KP + 16 * s + 8 * lg);
          st[kt] = mfma32<QF16>(a, qreg[s], st[kt]);
        }
      }

      // Scores in log2 units (ALiBi folded in); element r of subtile kt is key
      // n0 + 32 kt + 8 (r/4) + 4 lg + r%4.
      if constexpr (ALIBI) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int n = n0 + 32 * kt + 8 * (r >> 2) + 4 * lg + (r & 3);
            st[kt][r] = __builtin_fmaf(st[kt][r], c2, slope2 * (float)(n - m));
          }
      }
      // Masked entries at -inf; only tiles that cross the diagonal, the window
      // edge or the sequence end pay for it (one wave-uniform branch).
      bool need_mask = n0 + C::BN > S;
      if constexpr (MASK != MASK_NONE) need_mask = need_mask || (n0 + C::BN - 1 > mw);
      if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (n0 <= mw + 31 - W);
      if (need_mask) {
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int n = n0 + 32 * kt + 8 * (r >> 2) + 4 * lg + (r & 3);
            bool ok = n < S;
            if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
            if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
            st[kt][r] = ok ? st[kt][r] : -INFINITY;
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
      if (__any(m_new > m_run + 8.f)) {   // raise the reference max (wave-uniform)
        const float alpha = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int i = 0; i < C::MT; ++i) acc[i] *= alpha;
        m_run = m_new;
      }
      const float m_use = (m_run == -INFINITY) ? 0.f : m_run;

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
      l_run += rs;

      // O^T += V^T P^T; the V^T operand is two transpose reads of row-major V.
      // The head-dimension tiles are independent accumulators, interleaved.
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
#pragma unroll
          for (int mt = 0; mt < C::MT; ++mt) {
            const uint16_t* base = Vs + (32 * kt + 16 * hf + tr_key) * C::VP + 32 * mt + tr_col;
            const u32x2 lo = lds_read_tr16(base);
            const u32x2 hi = lds_read_tr16(base + 8 * C::VP);
            const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
            acc[mt] = mfma32(a, pb[kt][hf], acc[mt]);
          }
        }
      }
    }

    if (more) {
      uint16_t* Kn = smem + ((t + 1 - t_begin) & 1) * C::STAGE;
      tile_commit<D, ROPE>(R, Kn, Kn + C::K_ELEMS, tid);
    }
    __syncthreads();
  }

  // Epilogue: O = acc / l, LSE = (m + log2 l) ln 2.
  const float l_tot = pair_sum(l_run);
  if (m < S) {
    const float inv = (l_tot > 0.f) ? 1.f / l_tot : 0.f;
    uint16_t* O = static_cast<uint16_t*>(p.o) + (bh * S + m) * D;
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) {
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        u32x2 w = {pack_bf16(acc[mt][4 * a] * inv, acc[mt][4 * a + 1] * inv),
                   pack_bf16(acc[mt][4 * a + 2] * inv, acc[mt][4 * a + 3] * inv)};
        *reinterpret_cast<u32x2*>(O + 32 * mt + 8 * a + 4 * lg) = w;
      }
    }
    if (lg == 0) p.lse[bh * S + m] = (l_tot > 0.f) ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
  }
}

template <int D, int ROPE, int MASK, bool ALIBI>
static int launch_one(const FwdParams& p0, hipStream_t st) {
  using C = TileCfg<D, ROPE>;
  FwdParams p = p0;
  p.heads_per_wg = heads_per_wg(p.H / p.Hkv);
  const int P = C::ROWS / p.heads_per_wg;
  const long long blocks = (long long)((p.S + P - 1) / P) * p.B * p.Hkv * ((p.H / p.Hkv) / p.heads_per_wg);
  hipLaunchKernelGGL((fwd_bf16_kernel<D, ROPE, MASK, ALIBI>), dim3((unsigned)blocks), dim3(C::THREADS), 0, st, p);
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
