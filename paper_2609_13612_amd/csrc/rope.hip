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
// the chunk pair (c, c + D/2); for interleaved a single chunk.
template <bool FP32, int D, int ROPE, bool INV>
__global__ __launch_bounds__(256) void rope_kernel(RopeParams p) {
  constexpr int E = FP32 ? 4 : 8;                                  // elements per 16-byte chunk
  constexpr int CPR = (ROPE == ROPE_NEOX) ? D / (2 * E) : D / E;   // items per row
  const long long idx = (long long)blockIdx.x * 256 + threadIdx.x;
  const long long per_b = (long long)p.S * CPR;
  const int nh = p.heads0 + p.heads1;
  const int ngroups = (nh + ROPE_HEADS_PER_THREAD - 1) / ROPE_HEADS_PER_THREAD;
  if (idx >= per_b * p.B * ngroups) return;
  const int item = (int)(idx % per_b);
  const long long rest = idx / per_b;
  const int b = (int)(rest % p.B), hg = (int)(rest / p.B);
  const int n = item / CPR, c = item % CPR;
  const int h_begin = hg * ROPE_HEADS_PER_THREAD;
  const int h_end = min(nh, h_begin + ROPE_HEADS_PER_THREAD);
  const float2* __restrict__ cs = p.table + (size_t)n * (D / 2) + ((ROPE == ROPE_NEOX) ? E * c : (E / 2) * c);

#pragma unroll 4
  for (int hh = h_begin; hh < h_end; ++hh) {
    const bool first = hh < p.heads0;
    const int head = first ? hh : hh - p.heads0;
    const int nheads = first ? p.heads0 : p.heads1;
    const size_t row = ((size_t)(b * nheads + head) * p.S + n) * D;
    const char* X = static_cast<const char*>(first ? p.x0 : p.x1);
    char* Y = static_cast<char*>(first ? p.y0 : p.y1);
    constexpr int EB = FP32 ? 4 : 2;   // bytes per element
    if constexpr (ROPE == ROPE_NEOX) {
      const size_t oa = (row + (size_t)E * c) * EB, ob = (row + D / 2 + (size_t)E * c) * EB;
      if constexpr (FP32) {
        float4 a = *reinterpret_cast<const float4*>(X + oa), bb = *reinterpret_cast<const float4*>(X + ob);
        rotate_neox4_f32<INV>(a, bb, cs);
        *reinterpret_cast<float4*>(Y + oa) = a;
        *reinterpret_cast<float4*>(Y + ob) = bb;
      } else {
        u32x4 a = ld16(X + oa), bb = ld16(X + ob);
        rotate_neox8<INV>(a, bb, cs);
        st16(Y + oa, a);
        st16(Y + ob, bb);
      }
    } else {
      const size_t o = (row + (size_t)E * c) * EB;
      if constexpr (FP32) {
        float4 x = *reinterpret_cast<const float4*>(X + o);
        rotate_interleaved4_f32<INV>(x, cs);
        *reinterpret_cast<float4*>(Y + o) = x;
      } else {
        u32x4 x = ld16(X + o);
        rotate_interleaved8<INV>(x, cs);
        st16(Y + o, x);
      }
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
