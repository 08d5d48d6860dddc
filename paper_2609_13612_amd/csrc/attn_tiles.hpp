// Key-tile staging shared by the forward and the dQ kernel: a 64-key tile of
// K (RoPE-rotated, rounded to fp16 under RoPE) and V is loaded from HBM into
// registers one tile ahead, then rotated and committed to one of two LDS
// stages.  K' rows use a pitch of D + 8 elements (16-byte reads by 32 rows
// fall in distinct banks); V rows use D + 16 (the four rows a transpose read
// touches fall in distinct banks).
#pragma once
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
  // staging work items: NeoX rotates chunk pairs (c, c + D/2); otherwise single chunks
  static constexpr int K_UNITS = (ROPE == ROPE_NEOX) ? D / 16 : D / 8;
  static constexpr int K_ITEMS = BN * K_UNITS;
  static constexpr int KPT = (K_ITEMS + THREADS - 1) / THREADS;
  static constexpr int V_ITEMS = BN * (D / 8);
  static constexpr int VPT = (V_ITEMS + THREADS - 1) / THREADS;
  static constexpr int CS = (ROPE == ROPE_NEOX) ? 4 : (ROPE == ROPE_INTERLEAVED ? 2 : 1);   // float4 per item
};

// Registers holding one key tile between its global load and its LDS commit.
template <int D, int ROPE>
struct TileRegs {
  using C = TileCfg<D, ROPE>;
  u32x4 ka[C::KPT];
  u32x4 kb[(ROPE == ROPE_NEOX) ? C::KPT : 1];
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
    R.ka[i] = ld16(K + (size_t)n * D + 8 * c);
    if constexpr (ROPE == ROPE_NEOX) {
      R.kb[i] = ld16(K + (size_t)n * D + D / 2 + 8 * c);
      load_cs(R.cs[i], table + (size_t)n * (D / 2) + 8 * c);
    } else if constexpr (ROPE == ROPE_INTERLEAVED) {
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
      u32x4 a = R.ka[i], bb = R.kb[i];
      rotate_neox8<false, true>(a, bb, R.cs[i]);
      *reinterpret_cast<u32x4*>(Ks + r * C::KP + 8 * c) = a;
      *reinterpret_cast<u32x4*>(Ks + r * C::KP + D / 2 + 8 * c) = bb;
    } else {
      u32x4 a = R.ka[i];
      if constexpr (ROPE == ROPE_INTERLEAVED) rotate_interleaved8<false, true>(a, R.cs[i]);
      *reinterpret_cast<u32x4*>(Ks + r * C::KP + 8 * c) = a;
    }
  }
}

template <int D, int ROPE>
__device__ __forceinline__ void tile_commit_v(const TileRegs<D, ROPE>& R, uint16_t* __restrict__ Vs, int tid) {
  using C = TileCfg<D, ROPE>;
#pragma unroll
  for (int i = 0; i < C::VPT; ++i) {
    const int it = tid + C::THREADS * i;
    if (C::V_ITEMS % C::THREADS != 0 && it >= C::V_ITEMS) break;
    const int r = it / (D / 8), c = it % (D / 8);
    *reinterpret_cast<u32x4*>(Vs + r * C::VP + 8 * c) = R.v[i];
  }
}

template <int D, int ROPE>
__device__ __forceinline__ void tile_commit(TileRegs<D, ROPE>& R, uint16_t* __restrict__ Ks,
                                            uint16_t* __restrict__ Vs, int tid) {
  tile_commit_k<D, ROPE>(R, Ks, tid);
  tile_commit_v<D, ROPE>(R, Vs, tid);
}

// Query heads packed per workgroup by the forward and the dQ kernel: the
// largest power of two <= 8 dividing the GQA group size.
inline int heads_per_wg(int G) {
  int hp = 1;
  while (hp < 8 && G % (2 * hp) == 0) hp *= 2;
  return hp;
}

}  // namespace af
