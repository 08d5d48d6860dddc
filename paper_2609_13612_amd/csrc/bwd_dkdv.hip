// dK/dV pass of the bf16 backward: pass 3 of the backward described in
// bwd_bf16.hip (Section 4.4), which launches it after the dQ pass.  Its
// kernels live in a translation unit of their own so that the build can give
// them their own code-generation options.
#include <type_traits>

#include "bwd_common.hpp"

namespace af {

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

// ---------------------------------------------------------------- launch
namespace {
struct DkdvPass {
  template <int D, int ROPE, int MASK, bool ALIBI, int EXT>
  static int run(const BwdParams& p, hipStream_t st) {
    using QC = QTileCfg<D>;
    const int nkb = (p.S + QC::KEYS - 1) / QC::KEYS;
    const dim3 grid((unsigned)(nkb * p.B * p.Hkv)), block(QC::THREADS);
    if (EXT == EXT_NONE && p.bk_ptr)
      hipLaunchKernelGGL((bwd_dkdv_kernel<D, ROPE, MASK, ALIBI, true>), grid, block, 0, st, p);
    else
      hipLaunchKernelGGL((bwd_dkdv_kernel<D, ROPE, MASK, ALIBI, false, EXT>), grid, block, 0, st, p);
    return hipGetLastError() == hipSuccess ? 0 : -3;
  }
};
}  // namespace

int launch_bwd_dkdv_bf16(int D, int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  return bwd_dispatch<DkdvPass>(D, rope, mask, alibi, ext, p, st);
}

}  // namespace af
