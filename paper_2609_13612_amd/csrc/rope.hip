// Standalone RoPE rotation (the separate pre-rotation path) and the cos/sin
// table every RoPE kernel reads.
//
// Pre-rotation (Section 5.3, the Rotation Calculus) reads Q and K and writes
// Q' and K' once: a pure HBM round trip, so this kernel is written for
// bandwidth: one launch covers both tensors, 16-byte vector loads and stores,
// consecutive threads walk consecutive 16-byte chunks of a row, and each
// thread reuses one position's cos/sin entries across a group of heads.
#include "common.hpp"
#include "launch.hpp"

namespace af {

// ---------------------------------------------------------------- table
// T[n][i] = (cos(n * omega_i), sin(n * omega_i)), omega_i = theta^(-2i/D),
// computed in fp64 and rounded once to fp32.
__global__ void rope_table_kernel(float2* __restrict__ T, int rows, int D, double theta) {
  const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const int half = D / 2;
  if (idx >= (long long)rows * half) return;
  const int n = (int)(idx / half), i = (int)(idx % half);
  const double w = pow(theta, -2.0 * (double)i / (double)D);
  const double a = (double)n * w;
  T[idx] = make_float2((float)cos(a), (float)sin(a));
}

int launch_rope_table(float2* table, int rows, int D, double theta, hipStream_t st) {
  const long long n = (long long)rows * (D / 2);
  const unsigned blocks = (unsigned)((n + 255) / 256);
  hipLaunchKernelGGL(rope_table_kernel, dim3(blocks), dim3(256), 0, st, table, rows, D, theta);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// ---------------------------------------------------------------- fp32 chunks
template <bool INV>
__device__ __forceinline__ void rotate_neox4_f32(float4& a, float4& b, const float2* __restrict__ cs) {
  const float4* t = reinterpret_cast<const float4*>(cs);
  float4 t0 = t[0], t1 = t[1];
  rotate_pair<INV>(a.x, b.x, t0.x, t0.y);
  rotate_pair<INV>(a.y, b.y, t0.z, t0.w);
  rotate_pair<INV>(a.z, b.z, t1.x, t1.y);
  rotate_pair<INV>(a.w, b.w, t1.z, t1.w);
}

template <bool INV>
__device__ __forceinline__ void rotate_interleaved4_f32(float4& x, const float2* __restrict__ cs) {
  const float4 t = *reinterpret_cast<const float4*>(cs);
  rotate_pair<INV>(x.x, x.y, t.x, t.y);
  rotate_pair<INV>(x.z, x.w, t.z, t.w);
}

// ---------------------------------------------------------------- rotation
constexpr int ROPE_HEADS_PER_THREAD = 8;

// Thread item: (head group, batch, position n, chunk c).  For NeoX an item is
// the chunk pair (c, c + D/2); for interleaved a single chunk.  A thread loads
// its cos/sin entries once, issues the loads of all its heads before rotating
// any of them (memory-level parallelism), then stores.
template <bool FP32, int D, int ROPE, bool INV>
__global__ __launch_bounds__(256) void rope_kernel(RopeParams p) {
  constexpr int E = FP32 ? 4 : 8;                                  // elements per 16-byte chunk
  constexpr int CPR = (ROPE == ROPE_NEOX) ? D / (2 * E) : D / E;   // items per row
  constexpr int HPT = ROPE_HEADS_PER_THREAD;
  constexpr int NCH = (ROPE == ROPE_NEOX) ? 2 : 1;                 // chunks per item
  constexpr int NT = (ROPE == ROPE_NEOX) ? E / 2 : E / 4;          // float4 of cos/sin per item
  constexpr int EB = FP32 ? 4 : 2;                                 // bytes per element
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long per_b = (long long)p.S * CPR;
  const int nh = p.heads0 + p.heads1;
  const int ngroups = (nh + HPT - 1) / HPT;
  if (idx >= per_b * p.B * ngroups) return;
  const int item = (int)(idx % per_b);
  const long long rest = idx / per_b;
  const int b = (int)(rest % p.B), hg = (int)(rest / p.B);
  const int n = item / CPR, c = item % CPR;
  const int h_begin = hg * HPT;

  float4 t[NT];
  load_cs(t, p.table + (size_t)n * (D / 2) + ((ROPE == ROPE_NEOX) ? E * c : (E / 2) * c));
  const size_t off0 = (size_t)n * D + (size_t)E * c;             // element offset of chunk 0 in the row
  const size_t off1 = off0 + D / 2;                               // NeoX partner chunk

  u32x4 x[HPT][NCH];
#pragma unroll
  for (int j = 0; j < HPT; ++j) {
    const int hh = min(h_begin + j, nh - 1);   // clamped: the surplus lanes' results are not stored
    const bool first = hh < p.heads0;
    const int head = first ? hh : hh - p.heads0;
    const size_t base = (size_t)(b * (first ? p.heads0 : p.heads1) + head) * p.S * D;
    const char* X = static_cast<const char*>(first ? p.x0 : p.x1);
    x[j][0] = ld16(X + (base + off0) * EB);
    if constexpr (NCH == 2) x[j][1] = ld16(X + (base + off1) * EB);
  }
#pragma unroll
  for (int j = 0; j < HPT; ++j) {
    if constexpr (FP32) {
      float4 a = __builtin_bit_cast(float4, x[j][0]);
      if constexpr (ROPE == ROPE_NEOX) {
        float4 bb = __builtin_bit_cast(float4, x[j][1]);
        rotate_neox4_f32<INV>(a, bb, reinterpret_cast<const float2*>(t));
        x[j][1] = __builtin_bit_cast(u32x4, bb);
      } else {
        rotate_interleaved4_f32<INV>(a, reinterpret_cast<const float2*>(t));
      }
      x[j][0] = __builtin_bit_cast(u32x4, a);
    } else {
      if constexpr (ROPE == ROPE_NEOX) rotate_neox8<INV>(x[j][0], x[j][1], t);
      else rotate_interleaved8<INV>(x[j][0], t);
    }
  }
#pragma unroll
  for (int j = 0; j < HPT; ++j) {
    const int hh = h_begin + j;
    if (hh < nh) {
      const bool first = hh < p.heads0;
      const int head = first ? hh : hh - p.heads0;
      const size_t base = (size_t)(b * (first ? p.heads0 : p.heads1) + head) * p.S * D;
      char* Y = static_cast<char*>(first ? p.y0 : p.y1);
      st16(Y + (base + off0) * EB, x[j][0]);
      if constexpr (NCH == 2) st16(Y + (base + off1) * EB, x[j][1]);
    }
  }
}

template <bool FP32, int D, int ROPE, bool INV>
static int launch_rope_one(const RopeParams& p, hipStream_t st) {
  constexpr int E = FP32 ? 4 : 8;
  constexpr int CPR = (ROPE == ROPE_NEOX) ? D / (2 * E) : D / E;
  const int nh = p.heads0 + p.heads1;
  const long long ngroups = (nh + ROPE_HEADS_PER_THREAD - 1) / ROPE_HEADS_PER_THREAD;
  const long long total = (long long)p.S * CPR * p.B * ngroups;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL((rope_kernel<FP32, D, ROPE, INV>), dim3(blocks), dim3(256), 0, st, p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <bool FP32, int D>
static int rope_dispatch(int rope, bool inverse, const RopeParams& p, hipStream_t st) {
  if (rope == ROPE_NEOX)
    return inverse ? launch_rope_one<FP32, D, ROPE_NEOX, true>(p, st) : launch_rope_one<FP32, D, ROPE_NEOX, false>(p, st);
  if (rope == ROPE_INTERLEAVED)
    return inverse ? launch_rope_one<FP32, D, ROPE_INTERLEAVED, true>(p, st)
                   : launch_rope_one<FP32, D, ROPE_INTERLEAVED, false>(p, st);
  return -2;
}

int launch_rope(bool fp32, int D, int rope, bool inverse, const RopeParams& p, hipStream_t st) {
  if (fp32) {
    if (D == 64) return rope_dispatch<true, 64>(rope, inverse, p, st);
    if (D == 128) return rope_dispatch<true, 128>(rope, inverse, p, st);
  } else {
    if (D == 64) return rope_dispatch<false, 64>(rope, inverse, p, st);
    if (D == 128) return rope_dispatch<false, 128>(rope, inverse, p, st);
  }
  return -2;
}

}  // namespace af
