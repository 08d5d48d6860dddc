// Device helpers shared by the gfx950 kernels: vector types, bf16 packing,
// the 32x32x16 bf16 MFMA, wave-level lane swaps, and the RoPE pair rotation.
//
// MFMA register layout used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   * A operand (32 x 16): lane l supplies row (l % 32) and 8 k-values;
//   * B operand (16 x 32): lane l supplies column (l % 32) and 8 k-values;
//     the lane group g = l / 32 selects which 8 of the 16 k-values, and A and B
//     use the same (g, element) -> k assignment, so a contraction only needs
//     both operands to list their k-values in the same order;
//   * C/D (32 x 32, 16 floats per lane): element r of lane l is
//     row 8*(r/4) + 4*(l/32) + (r%4), column l % 32.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace af {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

enum RopeKind { ROPE_NONE = 0, ROPE_NEOX = 1, ROPE_INTERLEAVED = 2 };
enum MaskKind { MASK_NONE = 0, MASK_CAUSAL = 1, MASK_SLIDING_WINDOW = 2 };

// ---------------------------------------------------------------- bf16 <-> fp32
__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round two floats to bf16 (nearest even) and pack: a in the low half.
__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
  f32x2 v = {a, b};
  bf16x2 r = __builtin_convertvector(v, bf16x2);
  return __builtin_bit_cast(uint32_t, r);
}

// Round two floats to fp16 (nearest even) and pack: a in the low half.
__device__ __forceinline__ uint32_t pack_f16(float a, float b) {
  f32x2 v = {a, b};
  f16x2 r = __builtin_convertvector(v, f16x2);
  return __builtin_bit_cast(uint32_t, r);
}

// Pack in the MFMA operand type: fp16 when F16, else bf16.
template <bool F16>
__device__ __forceinline__ uint32_t pack_op(float a, float b) {
  if constexpr (F16) return pack_f16(a, b);
  else return pack_bf16(a, b);
}

// ---------------------------------------------------------------- MFMA
// 32x32x16 MFMA with fp32 accumulation on bf16 (F16 = false) or fp16 operands.
template <bool F16 = false>
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  if constexpr (F16)
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  else
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Reductions over the lane pair (l, l ^ 32).  v_permlane32_swap exchanges the
// upper half of its first operand with the lower half of its second; with the
// same value in both, each lane ends up holding its own value in one result
// and its partner's in the other, so combining the two results reduces the pair.
__device__ __forceinline__ float pair_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ---------------------------------------------------------------- RoPE
// One pair (x_a, x_b) rotated by the angle whose cosine and sine are (c, s):
//   forward:  x_a' = x_a c - x_b s,   x_b' = x_a s + x_b c
//   inverse:  x_a' = x_a c + x_b s,   x_b' = -x_a s + x_b c   (rotation by -angle)
// Every kernel rotates through this one function (fp32 arithmetic from an
// fp32 cos/sin table); only the final rounding differs by destination.
template <bool INVERSE>
__device__ __forceinline__ void rotate_pair(float& xa, float& xb, float c, float s) {
  const float a = xa, b = xb;
  if (!INVERSE) {
    xa = __builtin_fmaf(a, c, -(b * s));
    xb = __builtin_fmaf(a, s, b * c);
  } else {
    xa = __builtin_fmaf(a, c, b * s);
    xb = __builtin_fmaf(-a, s, b * c);
  }
}

// NeoX: 8 consecutive pair indices i0..i0+7 whose first elements are the 8 bf16
// of `a` and whose partners (half a head away) are the 8 bf16 of `b`.
// t holds the (cos, sin) table entries of those 8 pairs for one position
// (t[j] = entries 2j and 2j+1).  The rotated values are rounded to fp16 when
// F16OUT (the attention kernels' rotated MFMA operands), else back to bf16
// (the rotation kernel's tensors).
template <bool INVERSE, bool F16OUT = false>
__device__ __forceinline__ void rotate_neox8(u32x4& a, u32x4& b, const float4 (&t)[4]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float a0 = bf_lo(a[w]), a1 = bf_hi(a[w]);
    float b0 = bf_lo(b[w]), b1 = bf_hi(b[w]);
    rotate_pair<INVERSE>(a0, b0, t[w].x, t[w].y);
    rotate_pair<INVERSE>(a1, b1, t[w].z, t[w].w);
    a[w] = pack_op<F16OUT>(a0, a1);
    b[w] = pack_op<F16OUT>(b0, b1);
  }
}

// NeoX run of 2W consecutive pair indices (V holds W words of two bf16 each:
// u32x2 for 4 pairs, u32x4 for 8), first elements in `a`, partners in `b`;
// t[w] holds the (cos, sin) entries of the word's two pairs, as in rotate_neox8.
template <bool INVERSE, bool F16OUT, typename V>
__device__ __forceinline__ void rotate_neox_run(V& a, V& b, const float4* t) {
  constexpr int W = sizeof(V) / sizeof(uint32_t);
#pragma unroll
  for (int w = 0; w < W; ++w) {
    float a0 = bf_lo(a[w]), a1 = bf_hi(a[w]);
    float b0 = bf_lo(b[w]), b1 = bf_hi(b[w]);
    rotate_pair<INVERSE>(a0, b0, t[w].x, t[w].y);
    rotate_pair<INVERSE>(a1, b1, t[w].z, t[w].w);
    a[w] = pack_op<F16OUT>(a0, a1);
    b[w] = pack_op<F16OUT>(b0, b1);
  }
}

// Interleaved: the 8 bf16 of `x` are 4 pairs (2i, 2i+1), i = i0..i0+3, with
// table entries t[0] = (i0, i0+1), t[1] = (i0+2, i0+3).
template <bool INVERSE, bool F16OUT = false>
__device__ __forceinline__ void rotate_interleaved8(u32x4& x, const float4 (&t)[2]) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    float a = bf_lo(x[w]), b = bf_hi(x[w]);
    const float c = (w & 1) ? t[w >> 1].z : t[w >> 1].x;
    const float sn = (w & 1) ? t[w >> 1].w : t[w >> 1].y;
    rotate_pair<INVERSE>(a, b, c, sn);
    x[w] = pack_op<F16OUT>(a, b);
  }
}

// Load N float4 = 2N consecutive (cos, sin) table entries.
template <int N>
__device__ __forceinline__ void load_cs(float4 (&t)[N], const float2* __restrict__ cs) {
  const float4* q = reinterpret_cast<const float4*>(cs);
#pragma unroll
  for (int j = 0; j < N; ++j) t[j] = q[j];
}

template <bool INVERSE, bool F16OUT = false>
__device__ __forceinline__ void rotate_neox8(u32x4& a, u32x4& b, const float2* __restrict__ cs) {
  float4 t[4];
  load_cs(t, cs);
  rotate_neox8<INVERSE, F16OUT>(a, b, t);
}

template <bool INVERSE, bool F16OUT = false>
__device__ __forceinline__ void rotate_interleaved8(u32x4& x, const float2* __restrict__ cs) {
  float4 t[2];
  load_cs(t, cs);
  rotate_interleaved8<INVERSE, F16OUT>(x, t);
}

// ---------------------------------------------------------------- global memory
__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

// Rotate a whole fp32 row in place (INVERSE: by the negative angle, the
// transpose of the rotation, which carries gradients back); cs holds the
// row's D/2 (cos, sin) pairs.  Used by the fp32 debug kernels.
template <int D, int ROPE, bool INVERSE = false>
__device__ __forceinline__ void rotate_row_f32(float* x, const float2* __restrict__ cs) {
  if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
    for (int i = 0; i < D / 2; ++i) rotate_pair<INVERSE>(x[i], x[i + D / 2], cs[i].x, cs[i].y);
  } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
    for (int i = 0; i < D / 2; ++i) rotate_pair<INVERSE>(x[2 * i], x[2 * i + 1], cs[i].x, cs[i].y);
  }
}

// gfx950 LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16
// lanes the sixteen 8-byte chunks the lanes address form a 4 x 16 matrix of
// 16-bit values (row r = the chunks of lanes 4r..4r+3, in lane order); lane i
// of the group receives column i, i.e. one value from each of the 4 rows.
__device__ __forceinline__ u32x2 lds_read_tr16(const uint16_t* p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  v4i16 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)(p));
  return __builtin_bit_cast(u32x2, r);
}

// XOR-swizzled LDS tiles.  A tile read both by rows (ds_read_b128: 16 lanes
// per cycle read the same 16-byte chunk of 16 consecutive rows) and
// transposed (ds_read_b64_tr_b16: 32 lanes per cycle read 64 bytes of 4
// consecutive rows) is stored unpadded, D elements per row, with the 16-byte
// chunk c of row r at chunk slot c ^ swz(r).  With 64 banks of 4 bytes, swz
// gives the 16 rows of a row read 16 different slots and the 4 rows of a
// transpose read disjoint groups of 4 slots, so both are conflict-free.
template <int D>
__device__ __forceinline__ int swz_chunk(int r) {
  static_assert(D == 64 || D == 128, "swizzle defined for D = 64 and 128");
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);      // 16 chunks per row
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);                  // 8 chunks, two rows per 256 B
}

// Element offset of (row r, column col) in a swizzled tile; col % 8 is kept,
// so 8-byte (and 16-byte, col % 8 == 0) accesses stay whole.
template <int D>
__device__ __forceinline__ int swz_at(int r, int col) {
  return r * D + ((((col >> 3) ^ swz_chunk<D>(r)) << 3) | (col & 7));
}

// Per-lane offsets into a swizzled tile for the MFMA operand reads, as a base
// and an XOR: swz depends on the row modulo 16 only, and the chunk's varying
// bits never overlap the lane's, so
//   row operand (lane = row r0 + l % 32, k-step k, 8 dims 16 k + 8 (l / 32)):
//     r0 * D + (row_base ^ 16 k)
//   transposed operand (rows r0 + 4 (l / 32) + (l % 16) / 4 (+8), columns
//     32 mt + 16 ((l / 16) % 2) + 4 (l % 4)), r0 a multiple of 16:
//     r0 * D + (tr_base[half] ^ 32 mt)
template <int D>
struct SwzLane {
  int row_base, tr_base[2];
  __device__ __forceinline__ explicit SwzLane(int lane) {
    const int lq = lane & 31, lg = lane >> 5;
    row_base = swz_at<D>(lq, 8 * lg);
    const int r = 4 * lg + ((lane & 15) >> 2), c = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    tr_base[0] = swz_at<D>(r, c);
    tr_base[1] = swz_at<D>(r + 8, c);
  }
  // A copy the compiler cannot see through: used inside a loop, it keeps the
  // per-read XORs there (one VALU each) instead of hoisting their results
  // into registers for the whole loop.
  __device__ __forceinline__ SwzLane opaque() const {
    SwzLane z = *this;
    asm volatile("" : "+v"(z.row_base), "+v"(z.tr_base[0]), "+v"(z.tr_base[1]));
    return z;
  }
};

// Swap bits 2 and 3 of a key (or query) index inside a block of 16.  P^T leaves
// the S^T MFMA with lane group g holding rows {8a + 4g + b}; storing the
// transposed operand with this permutation makes those 8 rows contiguous, so
// the PV-style MFMA reads them with one 16-byte LDS load.
__device__ __forceinline__ int perm16(int x) {
  return (x & ~0xC) | ((x & 0x8) >> 1) | ((x & 0x4) << 1);
}

}  // namespace af
