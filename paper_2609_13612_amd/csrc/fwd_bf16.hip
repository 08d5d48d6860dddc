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
//   workgroup = 8 waves (two per SIMD) = 256 query rows.  The rows are HP
//   query heads of one GQA group x 256/HP positions, so one rotated K tile
//   serves every head that reads it.  Each wave owns 32 query rows and walks
//   the key tiles (BN = 64 keys) as a two-stage software pipeline with one
//   barrier per tile: part A issues tile t+1's score MFMAs while the VALU
//   turns tile t's scores into probabilities (exp2, row sum, bf16 packing);
//   part B issues tile t's PV MFMAs while the VALU rotates and stages later
//   tiles and masks / reduces tile t+1's scores.  gfx950 issues MFMA and VALU
//   instructions of one wave concurrently when they are independent, so each
//   part keeps both units busy; a wave that stalls on LDS leaves its SIMD to
//   the other wave.  K' and V tiles are double-buffered in LDS (K'_{t+2} and
//   V_{t+1} are staged during iteration t, from registers loaded one
//   iteration earlier).
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
#include <type_traits>

#include "attn_tiles.hpp"
#include "launch.hpp"

namespace af {

template <int D, int ROPE, int MASK, bool ALIBI, bool SPARSE, int EXT = EXT_NONE>
__global__ __launch_bounds__(512) void fwd_bf16_kernel(FwdParams p) {
  using C = TileCfg<D, ROPE>;
  constexpr bool QF16 = ROPE != ROPE_NONE;
  constexpr bool TBIAS = EXT == EXT_BIAS || EXT == EXT_RELU_BIAS;   // dense bias tensor
  constexpr bool RELU = EXT == EXT_RELU || EXT == EXT_RELU_BIAS;    // P = max(s, 0), unnormalised
  // scores leave prepare already scaled (and biased); plain softmax scales in probs
  constexpr bool PRESCALED = ALIBI || TBIAS || RELU;
  // Relu weights are unnormalised (not bounded by 1): P and V go to the PV
  // MFMA as fp16 (2^-12 rounding of P instead of bf16's 2^-9).
  __shared__ __attribute__((aligned(16))) uint16_t smem[(SPARSE ? 4 : 2) * C::STAGE];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lq = lane & 31, lg = lane >> 5;
  const int S = p.S;
  // Workgroup -> (batch, K/V head, head group, position block).  The position
  // block is the slow index and runs backwards, so the longest causal blocks
  // start first; consecutive workgroups walk (batch, K/V head, head group), and
  // with that count a multiple of 8 every block of one K/V head lands on the
  // same XCD and shares its L2.
  const int HP = p.heads_per_wg;                 // query heads per workgroup
  const int G = p.H / p.Hkv;
  const int groups = G / HP;
  const int units = p.B * p.Hkv * groups;
  const int unit = blockIdx.x % units;
  const int hg = unit % groups, bg = unit / groups;
  const int b = bg / p.Hkv, g = bg % p.Hkv;
  int h, p0, mw, p_end;
  int kg = 0;                                    // block-sparse: this wave's key group
  if constexpr (SPARSE) {
    // One 64-row query block; wave = (head hh, row half rh, key group kg).
    // The 4 / HP key groups take turns over the block's list of active tiles.
    const int ksplit = 4 / HP;
    kg = wave % ksplit;
    const int rh = (wave / ksplit) & 1, hh = wave / (2 * ksplit);
    const int nqb = (S + C::BN - 1) / C::BN;
    const int slot = (int)(blockIdx.x / units);
    // under a causal or window mask the last blocks have the longest lists
    const int qb = (MASK == MASK_NONE) ? slot : nqb - 1 - slot;
    h = g * G + hg * HP + hh;
    p0 = qb * C::BN;
    mw = p0 + 32 * rh;
    p_end = min(p0 + C::BN, S);
  } else {
    const int WPH = C::NW / HP;                  // waves per head
    const int P = 32 * WPH;                      // positions per workgroup
    const int npb = (S + P - 1) / P;
    const int pb = npb - 1 - (int)(blockIdx.x / units);
    h = g * G + hg * HP + wave / WPH;
    p0 = pb * P;
    mw = p0 + 32 * (wave % WPH);                 // first query row of this wave
    p_end = min(p0 + P, S);
  }
  const int m = mw + lq;                         // this lane's query row

  const size_t bh = (size_t)b * p.H + h;
  const uint16_t* __restrict__ Q = static_cast<const uint16_t*>(p.q) + bh * S * D;
  const uint16_t* __restrict__ K = static_cast<const uint16_t*>(p.k) + (size_t)bg * S * D;
  const uint16_t* __restrict__ V = static_cast<const uint16_t*>(p.v) + (size_t)bg * S * D;

  const float c2 = p.scale * kLog2e;                          // score -> log2 units
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;   // ALiBi slope, log2 units
  const int W = p.window;

  const int ntiles = (S + C::BN - 1) / C::BN;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (p_end - 1) / C::BN + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, p0 - W + 1) / C::BN;
  // The tiles the workgroup visits, by position i: t_begin + i, or under a
  // block-sparse mask the ascending active key blocks of its query block
  // (within the same range).
  __shared__ std::conditional_t<SPARSE, TileList<false>, int> tl;
  int ntl = t_end - t_begin;   // (block-sparse: set once the query loads are in flight)
  auto tile_at = [&](int i) -> int {
    if constexpr (SPARSE) return __builtin_amdgcn_readfirstlane((int)tl.tile[i]);
    else return t_begin + i;
  };
  // LDS stage of the tile at position X (K' and V): X & 1, or under a
  // block-sparse mask the slot X of the key groups.  The index is wave-uniform
  // and kept opaque so per-read offsets fold into the LDS instructions.
  auto kst = [&](int X) { return smem + __builtin_amdgcn_readfirstlane(SPARSE ? X : (X & 1)) * C::STAGE; };
  auto vst = [&](int X) { return kst(X) + C::K_ELEMS; };

  // Query operand (B of S^T = K Q^T): lane holds row m, dims 16s + 8lg .. +7.
  // Rows past S load row S-1 (finite data; never stored).
  const int mc = min(m, S - 1);
  const float* __restrict__ brow = nullptr;      // this lane's row of the bias tensor
  if constexpr (TBIAS) brow = p.bias + b * p.bias_sb + h * p.bias_sh + mc * p.bias_sq;
  u32x4 qreg[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) qreg[s] = ld16(Q + (size_t)mc * D + 16 * s + 8 * lg);
  if constexpr (SPARSE)   // the staging slots serve as scratch: nothing is staged yet
    ntl = __builtin_amdgcn_readfirstlane(
        tile_list_of_row<C::THREADS>(tl, smem, p.bq_ptr, p.bk_idx, p0 / C::BN, ntiles, t_begin, t_end, tid));
  if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
    for (int s = 0; s < C::KS / 2; ++s)
      rotate_neox8<false, true>(qreg[s], qreg[s + C::KS / 2], p.table + (size_t)mc * (D / 2) + 16 * s + 8 * lg);
  } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      rotate_interleaved8<false, true>(qreg[s], p.table + (size_t)mc * (D / 2) + 8 * s + 4 * lg);
  }

  // Prologue: stage K' of the first two tiles and V of the first; load the
  // registers of the first in-loop commit (K' of the third, V of the second).
  TileRegs<D, ROPE> R;
  if constexpr (!SPARSE) {
    for (int X = 0; X < min(2, ntl); ++X) {
      tile_load<D, ROPE>(R, K, V, p.table, tile_at(X) * C::BN, S, tid);
      tile_commit_k<D, ROPE>(R, kst(X), tid);
      if (X == 0) tile_commit_v<D, ROPE, RELU>(R, vst(X), tid);
    }
    // Every global load so far has landed (the commits waited for theirs);
    // saying so explicitly keeps the compiler from guarding the loop's
    // query-operand MFMAs with waits on the staging loads issued in the loop.
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0), expcnt and lgkmcnt unconstrained
    if (2 < ntl) tile_load_k<D, ROPE>(R, K, p.table, tile_at(2) * C::BN, S, tid);
    if (1 < ntl) tile_load_v<D, ROPE>(R, V, tile_at(1) * C::BN, S, tid);
  }

  f32x16 acc[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) acc[i] = f32x16{};
  float m_run = -INFINITY;   // reference max of the row, log2 units
  float l_run = 0.f;         // this lane's partial row sum (relative to m_run)
  float m_new = -INFINITY;   // max of the scores in flight (with m_run)

  // Transpose-read addressing for the V^T operand (see lds_read_tr16): lane i
  // of each 16-lane group reads 4 dims of key (4 lg + i/4) [+8 for the second
  // read]; the group's 16 lanes cover 16 dims starting at 16 * ((lane/16) & 1).
  const int tr_key = 4 * lg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int k_lane = lq * C::KP + 8 * lg;          // this lane's K' read offset
  const int v_lane = tr_key * C::VP + tr_col;      // this lane's V transpose-read offset

  // S^T = K' Q'^T for one tile: two 32-key subtiles, chains interleaved.
  auto scores = [&](f32x16 (&sc)[2], const uint16_t* Ks) {
    const uint16_t* kb = Ks + k_lane;
    sc[0] = f32x16{};
    sc[1] = f32x16{};
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(kb + 32 * kt * C::KP + 16 * s);
        sc[kt] = mfma32<QF16>(a, qreg[s], sc[kt]);
      }
  };
  // O^T += V^T P^T for one tile; the head-dimension accumulators interleaved.
  auto pv = [&](const u32x4 (&pop)[2][2], const uint16_t* Vs) {
    const uint16_t* vb = Vs + v_lane;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) {
          const uint16_t* base = vb + (32 * kt + 16 * hf) * C::VP + 32 * mt;
          const u32x2 lo = lds_read_tr16(base);
          const u32x2 hi = lds_read_tr16(base + 8 * C::VP);
          const u32x4 a = {lo[0], lo[1], hi[0], hi[1]};
          acc[mt] = mfma32<RELU>(a, pop[kt][hf], acc[mt]);
        }
  };

  // Scores of tile t in log2 units (ALiBi folded in), masked entries at -inf,
  // and their max merged into m_new.  Element r of subtile kt is key
  // n0 + 32 kt + 8 (r/4) + (r%4) + 4 lg of query mw + lq; mask and bias tests
  // compare one per-lane offset against the element's constant part, so
  // nothing per element stays live across tiles.  A tile with no visible key
  // for this wave (at the edge of the workgroup's range) is fully masked and
  // contributes P = 0.  Under a causal or window mask a key past S is also past
  // the query (rows past S are never stored), so only the unmasked variant
  // tests the sequence end.
  const int lane_off = 4 * lg - lq;
  auto prepare = [&](f32x16 (&sc)[2], int i) {
    const int n0 = tile_at(i) * C::BN;
    const int dq = n0 - mw + lane_off;        // key - query of element offset 0
    if constexpr (ALIBI) {
      const float fb = slope2 * (float)dq;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float cr = (float)(32 * kt + 8 * (r >> 2) + (r & 3));
          sc[kt][r] = __builtin_fmaf(sc[kt][r], c2, __builtin_fmaf(slope2, cr, fb));
        }
    }
    if constexpr (TBIAS || RELU) {
      // relu works in natural units, the softmax in log2 units
      const float cs = RELU ? p.scale : c2;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        float bv[16] = {};
        if constexpr (TBIAS) load_bias16(bv, brow, n0 + 32 * kt, lg, S);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sc[kt][r] = __builtin_fmaf(sc[kt][r], cs, RELU ? bv[r] : bv[r] * kLog2e);
      }
    }
    bool need_mask;
    if constexpr (MASK == MASK_NONE) need_mask = n0 + C::BN > S;
    else need_mask = n0 + C::BN - 1 > mw;
    if constexpr (MASK == MASK_SLIDING_WINDOW) need_mask = need_mask || (n0 <= mw + 31 - W);
    if (need_mask) {   // wave-uniform: diagonal, window-edge and sequence-end tiles only
      const int de = n0 + 4 * lg - S;        // key - S of element offset 0
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int cr = 32 * kt + 8 * (r >> 2) + (r & 3);
          bool ok;
          if constexpr (MASK == MASK_NONE) ok = de < -cr;
          else ok = dq <= -cr;
          if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (dq + W > -cr);
          sc[kt][r] = ok ? sc[kt][r] : -INFINITY;
        }
    }
    if constexpr (!RELU) {
      float mx = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sc[kt][r]);
      mx = pair_max(mx);
      if constexpr (!PRESCALED) mx *= c2;
      m_new = fmaxf(m_run, mx);
    }
  };
  // Raise the reference max when a row's max grew by more than 2^8 (rare,
  // wave-uniform): the accumulated O and l are rescaled together.
  auto raise = [&]() {
    if constexpr (RELU) return;   // no running max
    if (__any(m_new > m_run + 8.f)) {
      const float alpha = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < C::MT; ++i) acc[i] *= alpha;
      m_run = m_new;
    }
  };
  // P = exp2(score - m_run) as bf16 B operands, and the row sum (relu
  // attention: P = max(score, 0), no sum).
  auto probs = [&](const f32x16 (&sc)[2], u32x4 (&pop)[2][2]) {
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    float rs = 0.f;
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      float pv_[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if constexpr (RELU) {
          pv_[r] = fmaxf(sc[kt][r], 0.f);
        } else {
          const float arg = PRESCALED ? (sc[kt][r] - m_use) : __builtin_fmaf(sc[kt][r], c2, -m_use);
          pv_[r] = fast_exp2(arg);
          rs += pv_[r];
        }
      }
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int w = 0; w < 4; ++w) pop[kt][hf][w] = pack_op<RELU>(pv_[8 * hf + 2 * w], pv_[8 * hf + 2 * w + 1]);
    }
    l_run += rs;
  };

  // Materialise P and the row sum here: otherwise the compiler sinks their
  // computation next to the PV MFMAs that consume them, out of part A.
  auto pin_values = [](u32x4 (&pp)[2][2], float& l) {
    asm volatile("" : "+v"(pp[0][0]), "+v"(pp[0][1]), "+v"(pp[1][0]), "+v"(pp[1][1]), "+v"(l));
  };

  u32x4 pop[2][2];
  if constexpr (SPARSE) {
    // Block-sparse: each round the workgroup commits the next 4 / HP tiles of
    // the list into their own slots and then every wave computes the slot of
    // its key group: scores, mask and max, softmax, PV in sequence (the other
    // wave of the SIMD overlaps them).  The tiles travel through NR register
    // sets; the next round's first NR tiles are loaded before this round's
    // barrier, so their latency overlaps the compute.
    const int ksplit = 4 / HP;
    constexpr int NR = 2;
    TileRegs<D, ROPE> RS[NR];
    auto load_tile = [&](TileRegs<D, ROPE>& X, int pos) {
      tile_load<D, ROPE>(X, K, V, p.table, tile_at(pos) * C::BN, S, tid);
    };
#pragma unroll
    for (int j = 0; j < NR; ++j)
      if (j < min(ksplit, ntl)) load_tile(RS[j], j);
    f32x16 sc[2];
    for (int base = 0; base < ntl; base += ksplit) {
      const int nt = min(ksplit, ntl - base);   // wave-uniform
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (j < nt) {
          tile_commit<D, ROPE>(RS[j % NR], kst(j), vst(j), tid);
          if (j + NR < nt) load_tile(RS[j % NR], base + j + NR);
        }
      }
      const int next = base + ksplit, nt2 = min(ksplit, ntl - next);
#pragma unroll
      for (int j = 0; j < NR; ++j)
        if (j < nt2) load_tile(RS[j], next + j);
      __syncthreads();
      if (kg < nt && mw < S) {   // wave-uniform
        scores(sc, kst(kg));
        prepare(sc, base + kg);
        raise();
        probs(sc, pop);
        pv(pop, vst(kg));
      }
      __syncthreads();
    }
    // Merge the key groups' partial states (m, l, O) into key group 0: the
    // others hand theirs over through LDS, indexed [wave][element][lane].
    if (ksplit > 1) {
      constexpr int NE = 2 + 16 * C::MT;   // floats per lane: m, l, O
      static_assert(C::NW * NE * 64 * 4 <= 4 * C::STAGE * 2, "the merge reuses the four staging slots");
      float* xch = reinterpret_cast<float*>(smem);
      if (kg != 0) {
        float* dst = xch + wave * NE * 64 + lane;
        dst[0] = m_run;
        dst[64] = l_run;
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
          for (int r = 0; r < 16; ++r) dst[(2 + 16 * mt + r) * 64] = acc[mt][r];
      }
      __syncthreads();
      if (kg == 0) {
        float m_tot = m_run;
        for (int j = 1; j < ksplit; ++j) m_tot = fmaxf(m_tot, xch[(wave + j) * NE * 64 + lane]);
        const float a0 = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_tot);
        l_run *= a0;
#pragma unroll
        for (int mt = 0; mt < C::MT; ++mt) acc[mt] *= a0;
        for (int j = 1; j < ksplit; ++j) {
          const float* src = xch + (wave + j) * NE * 64 + lane;
          const float mj = src[0];
          const float aj = (mj == -INFINITY) ? 0.f : fast_exp2(mj - m_tot);
          l_run += aj * src[64];
#pragma unroll
          for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[mt][r] += aj * src[(2 + 16 * mt + r) * 64];
        }
        m_run = m_tot;
      }
    }
  } else {
    // Software pipeline, one barrier per tile.  Entering iteration t the
    // scores of tile t are prepared (masked, max merged, O rescaled).  Part A
    // issues tile t+1's score MFMAs together with tile t's exp2 / sum / bf16
    // packing; part B issues tile t's PV MFMAs together with staging (K'_{t+2}
    // rotated, V_{t+1}) and tile t+1's mask and max.  Within each part the
    // MFMA and VALU streams are independent, so every wave keeps the matrix
    // core and the vector ALU busy at once.  Tile X lives in LDS stage X & 1:
    // iteration t reads K'_{t+1} and V_t and writes K'_{t+2} and V_{t+1}, so
    // within an iteration no stage half is both read and written.
    f32x16 sa[2], sb[2];
    __syncthreads();
    if (ntl > 0) {
      scores(sa, kst(0));
      prepare(sa, 0);
      raise();
    }
    // The first iteration stages the third tile's K' into the stage just read.
    __syncthreads();
    int t = 0;   // position in the tile list
    auto iteration = [&](f32x16 (&cur)[2], f32x16 (&nxt)[2]) {
      // A
      probs(cur, pop);
      scores(nxt, kst(t + 1));
      pin_values(pop, l_run);   // keep the softmax work in this part
      // B.  Staging past the last tile rewrites a stage nobody reads any more
      // (clamped rows), which keeps this part free of branches.
      prepare(nxt, t + 1);
      pv(pop, vst(t));
      tile_commit_k<D, ROPE>(R, kst(t + 2), tid);
      tile_commit_v<D, ROPE, RELU>(R, vst(t + 1), tid);
      tile_load_k<D, ROPE>(R, K, p.table, tile_at(min(t + 3, ntl - 1)) * C::BN, S, tid);
      tile_load_v<D, ROPE>(R, V, tile_at(min(t + 2, ntl - 1)) * C::BN, S, tid);
      raise();
      __syncthreads();
      ++t;
    };
    // two iterations per trip so the score buffers alternate without copies
    while (t + 2 < ntl) {
      iteration(sa, sb);
      iteration(sb, sa);
    }
    if (t + 1 < ntl) {
      iteration(sa, sb);
      probs(sb, pop);
    } else if (t < ntl) {
      probs(sa, pop);
    }
    if (t < ntl) pv(pop, vst(t));
  }

  // Epilogue: O = acc / l, LSE = (m + log2 l) ln 2.  O leaves as whole rows
  // through the wave's rows of the staging memory, free once every wave is
  // past the key loop (store_rows_bf16).  Relu attention (unnormalised O, no
  // LSE) keeps each lane's own row stores: its key loop, which already
  // spills, ran 5 % slower with the staged store (the register allocation
  // moved), and the form below is the one it was measured fastest with.
  const float l_tot = pair_sum(l_run);
  if constexpr (RELU) {
    if (m < S && kg == 0) {
      const float inv = 1.f;
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
    }
  } else {
    const float inv = (l_tot > 0.f) ? 1.f / l_tot : 0.f;
    static_assert(C::NW * OUT_ROWS_ELEMS<D> <= (SPARSE ? 4 : 2) * C::STAGE, "the O rows fit the staging memory");
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt) acc[mt] *= inv;
    __syncthreads();
    if (kg == 0) {
      store_rows_bf16<D>(acc, smem + wave * OUT_ROWS_ELEMS<D>, static_cast<uint16_t*>(p.o) + (bh * S + mw) * D, S - mw,
                         lane);
      if (lg == 0 && m < S) p.lse[bh * S + m] = (l_tot > 0.f) ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
    }
  }
}

template <int D, int ROPE, int MASK, bool ALIBI, int EXT = EXT_NONE>
static int launch_one(const FwdParams& p0, hipStream_t st) {
  using C = TileCfg<D, ROPE>;
  FwdParams p = p0;
  const int G = p.H / p.Hkv;
  if (EXT == EXT_NONE && p.bq_ptr) {
    // block-sparse: one 64-row query block of up to 4 heads per workgroup
    p.heads_per_wg = heads_per_wg(G) < 4 ? heads_per_wg(G) : 4;
    const long long blocks = (long long)((p.S + C::BN - 1) / C::BN) * p.B * p.Hkv * (G / p.heads_per_wg);
    hipLaunchKernelGGL((fwd_bf16_kernel<D, ROPE, MASK, ALIBI, true>), dim3((unsigned)blocks), dim3(C::THREADS), 0, st,
                       p);
  } else {
    p.heads_per_wg = heads_per_wg(G);
    const int P = C::ROWS / p.heads_per_wg;
    const long long blocks = (long long)((p.S + P - 1) / P) * p.B * p.Hkv * (G / p.heads_per_wg);
    hipLaunchKernelGGL((fwd_bf16_kernel<D, ROPE, MASK, ALIBI, false, EXT>), dim3((unsigned)blocks), dim3(C::THREADS),
                       0, st, p);
  }
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <int D, int ROPE, int MASK>
static int dispatch_ext(bool alibi, int ext, const FwdParams& p, hipStream_t st) {
  switch (ext) {
    case EXT_NONE: return alibi ? launch_one<D, ROPE, MASK, true>(p, st) : launch_one<D, ROPE, MASK, false>(p, st);
    case EXT_BIAS: return launch_one<D, ROPE, MASK, false, EXT_BIAS>(p, st);
    case EXT_RELU: return launch_one<D, ROPE, MASK, false, EXT_RELU>(p, st);
    case EXT_RELU_BIAS: return launch_one<D, ROPE, MASK, false, EXT_RELU_BIAS>(p, st);
  }
  return -2;
}

template <int D, int ROPE>
static int dispatch_mask(int mask, bool alibi, int ext, const FwdParams& p, hipStream_t st) {
  switch (mask) {
    case MASK_NONE: return dispatch_ext<D, ROPE, MASK_NONE>(alibi, ext, p, st);
    case MASK_CAUSAL: return dispatch_ext<D, ROPE, MASK_CAUSAL>(alibi, ext, p, st);
    case MASK_SLIDING_WINDOW: return dispatch_ext<D, ROPE, MASK_SLIDING_WINDOW>(alibi, ext, p, st);
  }
  return -2;
}

template <int D>
static int dispatch_rope(int rope, int mask, bool alibi, int ext, const FwdParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return dispatch_mask<D, ROPE_NONE>(mask, alibi, ext, p, st);
    case ROPE_NEOX: return dispatch_mask<D, ROPE_NEOX>(mask, alibi, ext, p, st);
    case ROPE_INTERLEAVED: return dispatch_mask<D, ROPE_INTERLEAVED>(mask, alibi, ext, p, st);
  }
  return -2;
}

int launch_fwd_bf16(int D, int rope, int mask, bool alibi, int ext, const FwdParams& p, hipStream_t st) {
  if (ext != EXT_NONE && (alibi || p.bq_ptr)) return -2;   // not instantiated
  if (D == 64) return dispatch_rope<64>(rope, mask, alibi, ext, p, st);
  if (D == 128) return dispatch_rope<128>(rope, mask, alibi, ext, p, st);
  return -2;
}

}  // namespace af
