// Key-tile staging shared by the forward and the dQ kernel: a 64-key tile of
// K (RoPE-rotated, rounded to fp16 under RoPE) and V is loaded from HBM into
// registers one tile ahead, then rotated and committed to one of two LDS
// stages.  K' rows use a pitch of D + 8 elements (16-byte reads by 32 rows
// fall in distinct banks); V rows use D + 16 (the four rows a transpose read
// touches fall in distinct banks).
#pragma once
#include <type_traits>

#include "common.hpp"

namespace af {

template <int D, int ROPE>
struct TileCfg {
  static constexpr int NW = 8;                 // waves per workgroup
  static constexpr int THREADS = 64 * NW;
  static constexpr int ROWS = 32 * NW;         // query rows per workgroup
  static constexpr int BN = 64;                // keys per tile
  static constexpr int KS = D / 16;            // MFMA k-steps over the head dimension
  static constexpr int MT = D / 32;            // 32-row output tiles over the head dimension
  static constexpr int KP = D + 8;             // K tile pitch (elements): conflict-free 16-byte reads
  static constexpr int VP = D + 16;            // V tile pitch: conflict-free transpose reads
  static constexpr int K_ELEMS = BN * KP;
  static constexpr int V_ELEMS = BN * VP;
  static constexpr int STAGE = K_ELEMS + V_ELEMS;
  // staging work items: NeoX rotates pairs of KW-pair runs (dims [KW u, KW u + KW) with their
  // partners D/2 further on); otherwise single 8-element chunks.  At D = 64 a run is 4 pairs,
  // so the 64 rows give 512 items and every thread of the workgroup rotates one (with 8-pair
  // runs only half the waves would, and the barrier would wait for them).
  static constexpr int KW = (ROPE == ROPE_NEOX && D == 64) ? 4 : 8;
  static constexpr int K_UNITS = (ROPE == ROPE_NEOX) ? D / (2 * KW) : D / 8;
  static constexpr int K_ITEMS = BN * K_UNITS;
  static constexpr int KPT = (K_ITEMS + THREADS - 1) / THREADS;
  static constexpr int V_ITEMS = BN * (D / 8);
  static constexpr int VPT = (V_ITEMS + THREADS - 1) / THREADS;
  static constexpr int CS = (ROPE == ROPE_NEOX) ? KW / 2 : (ROPE == ROPE_INTERLEAVED ? 2 : 1);   // float4 per item
};

// Registers holding one key tile between its global load and its LDS commit
// (NeoX runs of 4 pairs travel as 8-byte halves).
template <int D, int ROPE>
struct TileRegs {
  using C = TileCfg<D, ROPE>;
  using KVec = std::conditional_t<C::KW == 4, u32x2, u32x4>;
  KVec ka[C::KPT];
  KVec kb[(ROPE == ROPE_NEOX) ? C::KPT : 1];
  float4 cs[C::KPT][C::CS];
  u32x4 v[C::VPT];
};

// Rows past S are clamped to row S-1 so every load is unconditional: those
// keys are masked out of the scores and their V rows (finite data) receive
// zero probability.  K and V halves can be loaded and committed separately.
template <int D, int ROPE>
__device__ __forceinline__ void tile_load_k(TileRegs<D, ROPE>& R, const uint16_t* __restrict__ K,
                                            const float2* __restrict__ table, int n0, int S, int tid) {
  using C = TileCfg<D, ROPE>;
#pragma unroll
  for (int i = 0; i < C::KPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::K_ITEMS % C::THREADS != 0 && it >= C::K_ITEMS) break;
    const int r = it / C::K_UNITS, c = it % C::K_UNITS, n = min(n0 + r, S - 1);
    if constexpr (ROPE == ROPE_NEOX) {
      using KV = typename TileRegs<D, ROPE>::KVec;
      R.ka[i] = *reinterpret_cast<const KV*>(K + (size_t)n * D + C::KW * c);
      R.kb[i] = *reinterpret_cast<const KV*>(K + (size_t)n * D + D / 2 + C::KW * c);
      load_cs(R.cs[i], table + (size_t)n * (D / 2) + C::KW * c);
    } else {
      R.ka[i] = ld16(K + (size_t)n * D + 8 * c);
    }
    if constexpr (ROPE == ROPE_INTERLEAVED) {
      load_cs(R.cs[i], table + (size_t)n * (D / 2) + 4 * c);
    }
  }
}

template <int D, int ROPE>
__device__ __forceinline__ void tile_load_v(TileRegs<D, ROPE>& R, const uint16_t* __restrict__ V, int n0, int S,
                                            int tid) {
  using C = TileCfg<D, ROPE>;
#pragma unroll
  for (int i = 0; i < C::VPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::V_ITEMS % C::THREADS != 0 && it >= C::V_ITEMS) break;
    const int r = it / (D / 8), c = it % (D / 8), n = min(n0 + r, S - 1);
    R.v[i] = ld16(V + (size_t)n * D + 8 * c);
  }
}

template <int D, int ROPE>
__device__ __forceinline__ void tile_load(TileRegs<D, ROPE>& R, const uint16_t* __restrict__ K,
                                          const uint16_t* __restrict__ V, const float2* __restrict__ table,
                                          int n0, int S, int tid) {
  tile_load_k<D, ROPE>(R, K, table, n0, S, tid);
  tile_load_v<D, ROPE>(R, V, n0, S, tid);
}

// Rotate the staged K rows and write K' (and, separately, V) into an LDS stage.
template <int D, int ROPE>
__device__ __forceinline__ void tile_commit_k(TileRegs<D, ROPE>& R, uint16_t* __restrict__ Ks, int tid) {
  using C = TileCfg<D, ROPE>;
#pragma unroll
  for (int i = 0; i < C::KPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::K_ITEMS % C::THREADS != 0 && it >= C::K_ITEMS) break;
    const int r = it / C::K_UNITS, c = it % C::K_UNITS;
    if constexpr (ROPE == ROPE_NEOX) {
      auto a = R.ka[i], bb = R.kb[i];
      rotate_neox_run<false, true>(a, bb, R.cs[i]);
      *reinterpret_cast<decltype(a)*>(Ks + r * C::KP + C::KW * c) = a;
      *reinterpret_cast<decltype(a)*>(Ks + r * C::KP + D / 2 + C::KW * c) = bb;
    } else {
      u32x4 a = R.ka[i];
      if constexpr (ROPE == ROPE_INTERLEAVED) rotate_interleaved8<false, true>(a, R.cs[i]);
      *reinterpret_cast<u32x4*>(Ks + r * C::KP + 8 * c) = a;
    }
  }
}

// V16: store V converted to fp16 (exact for |v| < 65504), for fp16 P operands.
template <int D, int ROPE, bool V16 = false>
__device__ __forceinline__ void tile_commit_v(const TileRegs<D, ROPE>& R, uint16_t* __restrict__ Vs, int tid) {
  using C = TileCfg<D, ROPE>;
#pragma unroll
  for (int i = 0; i < C::VPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::V_ITEMS % C::THREADS != 0 && it >= C::V_ITEMS) break;
    const int r = it / (D / 8), c = it % (D / 8);
    u32x4 v = R.v[i];
    if constexpr (V16) {
#pragma unroll
      for (int w = 0; w < 4; ++w) v[w] = pack_f16(bf_lo(v[w]), bf_hi(v[w]));
    }
    *reinterpret_cast<u32x4*>(Vs + r * C::VP + 8 * c) = v;
  }
}

template <int D, int ROPE, bool V16 = false>
__device__ __forceinline__ void tile_commit(TileRegs<D, ROPE>& R, uint16_t* __restrict__ Ks,
                                            uint16_t* __restrict__ Vs, int tid) {
  tile_commit_k<D, ROPE>(R, Ks, tid);
  tile_commit_v<D, ROPE, V16>(R, Vs, tid);
}

// ---------------------------------------------------------------- output rows
// Store a wave's 32 rows of a bf16 output held as MFMA accumulators (lane
// lq owns row lq; element 4 a + e of acc[mt] is column 32 mt + 8 a + 4 lg + e)
// through the wave's own 32 rows of LDS at a pitch of D + 8 elements
// (OUT_ROWS_ELEMS), so that every store instruction writes whole rows (64
// lanes x 16 bytes) instead of each lane writing its own row in pieces.  The
// padding keeps the row writes and the chunk reads within two bank passes
// with every address an immediate offset.  Rows from `rows` on are not
// stored.  The caller makes sure no other wave still reads the LDS region.
template <int D>
constexpr int OUT_ROWS_ELEMS = 32 * (D + 8);   // one wave's LDS rows (elements)

template <int D>
__device__ __forceinline__ void store_rows_bf16(const f32x16 (&acc)[D / 32], uint16_t* __restrict__ lds,
                                                uint16_t* __restrict__ dst, int rows, int lane) {
  constexpr int OP = D + 8;           // LDS row pitch (elements)
  constexpr int CPR = D / 8;          // 16-byte chunks per row
  constexpr int NCH = 32 * CPR / 64;  // chunks per lane
  const int lq = lane & 31, lg = lane >> 5;
#pragma unroll
  for (int mt = 0; mt < D / 32; ++mt)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      const u32x2 w = {pack_bf16(acc[mt][4 * a], acc[mt][4 * a + 1]), pack_bf16(acc[mt][4 * a + 2], acc[mt][4 * a + 3])};
      *reinterpret_cast<u32x2*>(lds + lq * OP + 32 * mt + 8 * a + 4 * lg) = w;
    }
  // (a wave's LDS accesses complete in order: the reads below see these writes)
  u32x4 ch[NCH];
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int c = lane + 64 * i;
    ch[i] = *reinterpret_cast<const u32x4*>(lds + (c / CPR) * OP + 8 * (c % CPR));
  }
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    const int c = lane + 64 * i, r = c / CPR;
    if (r < rows) *reinterpret_cast<u32x4*>(dst + (size_t)r * D + 8 * (c % CPR)) = ch[i];
  }
}

// ---------------------------------------------------------------- dense bias rows
// The 16 bias values a lane's score registers of one 32-key subtile need:
// keys k0 + 8 a + 4 lg + e of the bias row `row` into register 4 a + e.  Each
// group of four is consecutive in memory, so a subtile inside the sequence
// takes four 16-byte loads; at the sequence end each key is guarded (0 past S).
__device__ __forceinline__ void load_bias16(float (&bv)[16], const float* __restrict__ row, int k0, int lg, int S) {
  if (k0 + 32 <= S) {   // wave-uniform
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      float4 x;
      __builtin_memcpy(&x, row + k0 + 8 * a + 4 * lg, sizeof(x));   // 4-byte alignment is all a row guarantees
      bv[4 * a] = x.x;
      bv[4 * a + 1] = x.y;
      bv[4 * a + 2] = x.z;
      bv[4 * a + 3] = x.w;
    }
  } else {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int n = k0 + 8 * (r >> 2) + 4 * lg + (r & 3);
      bv[r] = (n < S) ? row[n] : 0.f;
    }
  }
}

// ---------------------------------------------------------------- block-sparse tile lists
// Largest number of 64-wide blocks along the sequence a block-sparse launch
// accepts (S <= 131072); the host rejects longer sequences.
constexpr int SPARSE_MAX_BLOCKS = 2048;

// LDS for one workgroup's list of active tiles: the block indices, ascending,
// and (for lists that merge several rows) which of the rows hold each block.
template <bool ROWS>
struct TileList {
  uint16_t tile[SPARSE_MAX_BLOCKS];
  uint8_t rows[SPARSE_MAX_BLOCKS];
};
template <>
struct TileList<false> {
  uint16_t tile[SPARSE_MAX_BLOCKS];
};
// LDS the list construction needs only while it runs (2080 bytes): a byte per
// block marking the rows that hold it, and one count per wave.
constexpr int TILE_LIST_SCRATCH_BYTES = SPARSE_MAX_BLOCKS + 8 * 4;

// The ascending union of the compressed rows r0 .. r0+nr-1 (nr <= 8) of a
// block mask (ptr [rows+1], idx: each row's active blocks), restricted to
// blocks in [lo, hi) (the range the elementwise mask can reach), with a bit
// per row saying which rows hold each block (stored only when ROWS).  Entries
// outside [lo, hi), which contains only valid blocks, are ignored, so a
// malformed mask cannot index outside the tiles.  ``scratch`` is TILE_LIST_SCRATCH_BYTES of 4-byte aligned LDS that is
// free until the call returns.  Every thread of the workgroup must call it; it
// returns the count after a barrier, and the list is then valid.
template <int THREADS, bool ROWS>
__device__ int build_tile_list(TileList<ROWS>& L, void* scratch, const int* __restrict__ ptr,
                               const int* __restrict__ idx, int r0, int nr, int nb, int lo, int hi, int tid) {
  uint32_t* member = static_cast<uint32_t*>(scratch);   // one byte per block
  int* wave_total = reinterpret_cast<int*>(member + SPARSE_MAX_BLOCKS / 4);
  for (int w = tid; w < (nb + 3) / 4; w += THREADS) member[w] = 0u;
  __syncthreads();
  for (int j = 0; j < nr; ++j) {
    const int e0 = ptr[r0 + j], e1 = ptr[r0 + j + 1];
    for (int e = e0 + tid; e < e1; e += THREADS) {
      const int b = idx[e];
      if (b >= lo && b < hi) atomicOr(&member[b >> 2], (1u << j) << (8 * (b & 3)));
    }
  }
  __syncthreads();
  // compaction: thread t owns blocks [t*per, (t+1)*per); its output position is
  // the number of active blocks owned by lower threads (a scan within the wave,
  // then the totals of the lower waves)
  static_assert(THREADS % 64 == 0 && THREADS <= 512, "whole waves, at most eight");
  const int per = (nb + THREADS - 1) / THREADS;
  auto byte_of = [&](int b) { return (member[b >> 2] >> (8 * (b & 3))) & 0xffu; };
  int cnt = 0;
  for (int b = tid * per; b < min(nb, (tid + 1) * per); ++b) cnt += byte_of(b) != 0u;
  const int lane = tid & 63, wave = tid >> 6;
  int incl = cnt;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int x = __shfl_up(incl, off, 64);
    if (lane >= off) incl += x;
  }
  if (lane == 63) wave_total[wave] = incl;
  __syncthreads();
  int pos = incl - cnt, total = 0;
#pragma unroll
  for (int w = 0; w < THREADS / 64; ++w) {
    const int x = wave_total[w];
    pos += (w < wave) ? x : 0;
    total += x;
  }
  for (int b = tid * per; b < min(nb, (tid + 1) * per); ++b) {
    const uint32_t m = byte_of(b);
    if (m != 0u) {
      L.tile[pos] = (uint16_t)b;
      if constexpr (ROWS) L.rows[pos] = (uint8_t)m;
      ++pos;
    }
  }
  __syncthreads();
  return total;
}

// The list of ONE compressed row r (restricted to [lo, hi)), read directly
// when the row is strictly ascending (the canonical form, which needs no
// sorting or duplicate removal): wave 0 streams the row, keeps the entries in
// range in order and checks the order on the way.  Any other row goes through
// build_tile_list.  ``scratch`` as there, plus 8 more bytes.  Every thread of
// the workgroup must call it; the list is valid when it returns.
template <int THREADS>
__device__ int tile_list_of_row(TileList<false>& L, void* scratch, const int* __restrict__ ptr,
                                const int* __restrict__ idx, int r, int nb, int lo, int hi, int tid) {
  int* res = reinterpret_cast<int*>(static_cast<char*>(scratch) + TILE_LIST_SCRATCH_BYTES);
  if (tid < 64) {
    const int e0 = ptr[r], e1 = ptr[r + 1];
    int n = 0;
    bool ordered = true;
    for (int e = e0 + tid; e - tid < e1; e += 64) {
      const bool live = e < e1;
      const int x = live ? idx[e] : 0;
      const int nxt = (e + 1 < e1) ? idx[e + 1] : 0x7fffffff;
      ordered = ordered && __ballot(live && x >= nxt) == 0ull;
      const bool in = live && x >= lo && x < hi;
      const unsigned long long bits = __ballot(in);
      const int pos = n + __popcll(bits & ((1ull << tid) - 1ull));
      if (in && pos < SPARSE_MAX_BLOCKS) L.tile[pos] = (uint16_t)x;
      n += __popcll(bits);
    }
    if (tid == 0) {
      res[0] = n;
      res[1] = ordered;
    }
  }
  __syncthreads();
  const int n = res[0], ordered = res[1];
  // every thread holds the result before anyone reuses the scratch memory
  // (the fallback below, or the caller's staging)
  __syncthreads();
  if (!ordered) return build_tile_list<THREADS>(L, scratch, ptr, idx, r, 1, nb, lo, hi, tid);
  return n;
}

// Query heads packed per workgroup by the forward and the dQ kernel: the
// largest power of two <= 8 dividing the GQA group size.
inline int heads_per_wg(int G) {
  int hp = 1;
  while (hp < 8 && G % (2 * hp) == 0) hp *= 2;
  return hp;
}

}  // namespace af
