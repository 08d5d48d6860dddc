// fp32 debug forward: the same method as the bf16 MFMA kernel (RoPE on the
// query once and on every staged key tile, post-matmul modifications, online
// softmax over key tiles, masked tiles skipped) in plain fp32 FMA arithmetic,
// one query row per thread.  It exists to check the method at fp32 precision,
// not for speed.
#include "common.hpp"
#include "launch.hpp"

namespace af {

constexpr int F32_ROWS = 64;   // query rows per workgroup (one wave)
constexpr int F32_BN = 32;     // keys per tile

template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(64) void fwd_fp32_kernel(FwdParams p) {
  __shared__ float Kf[F32_BN][D + 1];
  __shared__ float Vf[F32_BN][D + 1];
  const int tid = threadIdx.x;
  const int S = p.S;
  const int BH = p.B * p.H;
  const int nqb = (S + F32_ROWS - 1) / F32_ROWS;
  const int bh = blockIdx.x % BH;
  const int qb = nqb - 1 - (int)(blockIdx.x / BH);
  const int b = bh / p.H, h = bh % p.H;
  const int g = h / (p.H / p.Hkv);
  const int m0 = qb * F32_ROWS;
  const int m = m0 + tid;
  const float* __restrict__ Q = static_cast<const float*>(p.q) + (size_t)bh * S * D;
  const float* __restrict__ K = static_cast<const float*>(p.k) + (size_t)(b * p.Hkv + g) * S * D;
  const float* __restrict__ V = static_cast<const float*>(p.v) + (size_t)(b * p.Hkv + g) * S * D;

  float q[D], acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = (m < S) ? Q[(size_t)m * D + d] : 0.f;
    acc[d] = 0.f;
  }
  if (ROPE != ROPE_NONE && m < S) rotate_row_f32<D, ROPE>(q, p.table + (size_t)m * (D / 2));

  const float c2 = p.scale * kLog2e;
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;
  const int W = p.window;
  const int ntiles = (S + F32_BN - 1) / F32_BN;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (min(m0 + F32_ROWS, S) - 1) / F32_BN + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, m0 - W + 1) / F32_BN;

  float m_run = -INFINITY, l_run = 0.f;
  for (int t = t_begin; t < t_end; ++t) {
    const int n0 = t * F32_BN;
    __syncthreads();
    // Stage the tile: thread tid < F32_BN rotates key row n0 + tid.
    for (int r = 0; r < F32_BN; ++r) {
      const int n = n0 + r;
      for (int d = tid; d < D; d += 64) {
        Kf[r][d] = (n < S) ? K[(size_t)n * D + d] : 0.f;
        Vf[r][d] = (n < S) ? V[(size_t)n * D + d] : 0.f;
      }
    }
    __syncthreads();
    if (ROPE != ROPE_NONE && tid < F32_BN && n0 + tid < S) {
      float row[D];
#pragma unroll
      for (int d = 0; d < D; ++d) row[d] = Kf[tid][d];
      rotate_row_f32<D, ROPE>(row, p.table + (size_t)(n0 + tid) * (D / 2));
#pragma unroll
      for (int d = 0; d < D; ++d) Kf[tid][d] = row[d];
    }
    __syncthreads();
    if (m >= S) continue;

    float sc[F32_BN];
    float mx = -INFINITY;
    for (int j = 0; j < F32_BN; ++j) {
      const int n = n0 + j;
      float dot = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) dot = __builtin_fmaf(q[d], Kf[j][d], dot);
      float x = ALIBI ? __builtin_fmaf(dot, c2, slope2 * (float)(n - m)) : dot * c2;
      bool ok = n < S;
      if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
      if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
      sc[j] = ok ? x : -INFINITY;
      mx = fmaxf(mx, sc[j]);
    }
    const float m_new = fmaxf(m_run, mx);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = exp2f(m_run - m_use);
    l_run *= alpha;
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] *= alpha;
    for (int j = 0; j < F32_BN; ++j) {
      const float pj = exp2f(sc[j] - m_use);
      l_run += pj;
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] = __builtin_fmaf(pj, Vf[j][d], acc[d]);
    }
    m_run = m_new;
  }
  if (m < S) {
    const float inv = (l_run > 0.f) ? 1.f / l_run : 0.f;
    float* O = static_cast<float*>(p.o) + ((size_t)bh * S + m) * D;
#pragma unroll
    for (int d = 0; d < D; ++d) O[d] = acc[d] * inv;
    p.lse[(size_t)bh * S + m] = (l_run > 0.f) ? (m_run + log2f(l_run)) * kLn2 : -INFINITY;
  }
}

template <int D, int ROPE, int MASK, bool ALIBI>
static int launch_one(const FwdParams& p, hipStream_t st) {
  const int nqb = (p.S + F32_ROWS - 1) / F32_ROWS;
  hipLaunchKernelGGL((fwd_fp32_kernel<D, ROPE, MASK, ALIBI>), dim3((unsigned)(nqb * p.B * p.H)), dim3(64), 0, st, p);
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

int launch_fwd_fp32(int D, int rope, int mask, bool alibi, const FwdParams& p, hipStream_t st) {
  if (D == 64) return dispatch_rope<64>(rope, mask, alibi, p, st);
  if (D == 128) return dispatch_rope<128>(rope, mask, alibi, p, st);
  return -2;
}

}  // namespace af
