// Helpers shared by the two gradient passes of the bf16 backward (the dQ pass
// in bwd_bf16.hip, the dK/dV pass in bwd_dkdv.hip): row operands, gradient
// stores through the inverse rotation, transposed and swizzled LDS operands,
// and the dispatch from runtime variant arguments to kernel instantiations.
#pragma once
#include "attn_tiles.hpp"
#include "launch.hpp"

namespace af {

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

// ---------------------------------------------------------------- dispatch
// Map the runtime variant (D, rope, mask, alibi, ext) to Pass::run<D, ROPE,
// MASK, ALIBI, EXT>(p, st).  Extensions other than EXT_NONE are instantiated
// only without ALiBi and block masks; anything else returns -2.
template <class Pass, int D, int ROPE, int MASK>
int bwd_dispatch_ext(bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  switch (ext) {
    case EXT_NONE:
      return alibi ? Pass::template run<D, ROPE, MASK, true, EXT_NONE>(p, st)
                   : Pass::template run<D, ROPE, MASK, false, EXT_NONE>(p, st);
    case EXT_BIAS: return Pass::template run<D, ROPE, MASK, false, EXT_BIAS>(p, st);
    case EXT_RELU: return Pass::template run<D, ROPE, MASK, false, EXT_RELU>(p, st);
    case EXT_RELU_BIAS: return Pass::template run<D, ROPE, MASK, false, EXT_RELU_BIAS>(p, st);
  }
  return -2;
}

template <class Pass, int D, int ROPE>
int bwd_dispatch_mask(int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  switch (mask) {
    case MASK_NONE: return bwd_dispatch_ext<Pass, D, ROPE, MASK_NONE>(alibi, ext, p, st);
    case MASK_CAUSAL: return bwd_dispatch_ext<Pass, D, ROPE, MASK_CAUSAL>(alibi, ext, p, st);
    case MASK_SLIDING_WINDOW: return bwd_dispatch_ext<Pass, D, ROPE, MASK_SLIDING_WINDOW>(alibi, ext, p, st);
  }
  return -2;
}

template <class Pass, int D>
int bwd_dispatch_rope(int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return bwd_dispatch_mask<Pass, D, ROPE_NONE>(mask, alibi, ext, p, st);
    case ROPE_NEOX: return bwd_dispatch_mask<Pass, D, ROPE_NEOX>(mask, alibi, ext, p, st);
    case ROPE_INTERLEAVED: return bwd_dispatch_mask<Pass, D, ROPE_INTERLEAVED>(mask, alibi, ext, p, st);
  }
  return -2;
}

template <class Pass>
int bwd_dispatch(int D, int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st) {
  if (ext != EXT_NONE && (alibi || p.bq_ptr || p.bk_ptr)) return -2;   // not instantiated
  if (D == 64) return bwd_dispatch_rope<Pass, 64>(rope, mask, alibi, ext, p, st);
  if (D == 128) return bwd_dispatch_rope<Pass, 128>(rope, mask, alibi, ext, p, st);
  return -2;
}

}  // namespace af
