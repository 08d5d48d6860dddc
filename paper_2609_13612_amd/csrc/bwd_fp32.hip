// fp32 debug backward: the same three passes as the bf16 backward (Section
// 4.4: row statistics; dK/dV over query tiles with the GQA group's heads
// summed; dQ over key tiles; no atomics), in plain fp32 FMA arithmetic with one
// row per thread and the rotation recomputed on every staged tile.  It exists
// to check the backward at fp32 precision, not for speed.
//
// With s_ij = scale <R_i q_i, R_j k_j> + bias_ij and P the softmax rows:
//   dV_j  = sum_i P_ij dO_i
//   dP_ij = <dO_i, v_j>,  delta_i = sum_d dO_id O_id,  dS_ij = P_ij (dP_ij - delta_i)
//   dQ_i  = R_i^T (scale sum_j dS_ij R_j k_j),  dK_j = R_j^T (scale sum_i dS_ij R_i q_i)
// P_ij is re-derived from the forward's LSE: P_ij = exp(s_ij - LSE_i).
#include "common.hpp"
#include "launch.hpp"

namespace af {

constexpr int B32_ROWS = 64;   // rows per workgroup (one wave)
constexpr int B32_BT = 32;     // rows per staged tile

// delta_i and LSE_i in log2 units (+inf for an empty row, so its P is 0).
__global__ void bwd_fp32_prep_kernel(BwdParams p, int D) {
  const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long long)p.B * p.H * p.S) return;
  const float* __restrict__ dO = static_cast<const float*>(p.dout) + i * D;
  const float* __restrict__ O = static_cast<const float*>(p.o) + i * D;
  float s = 0.f;
  for (int d = 0; d < D; ++d) s = __builtin_fmaf(dO[d], O[d], s);
  p.delta[i] = s;
  const float l = p.lse[i];
  p.lse2[i] = (l == -INFINITY) ? INFINITY : l * kLog2e;
}

// One query row per thread: loops over the visible key tiles, each staged in
// LDS with K rotated by the first B32_BT threads.
template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(64) void bwd_fp32_dq_kernel(BwdParams p) {
  __shared__ float Kf[B32_BT][D + 1];
  __shared__ float Vf[B32_BT][D + 1];
  const int tid = threadIdx.x;
  const int S = p.S;
  const int BH = p.B * p.H;
  const int bh = blockIdx.x % BH;
  const int qb = (int)(blockIdx.x / BH);
  const int b = bh / p.H, h = bh % p.H;
  const int g = h / (p.H / p.Hkv);
  const int m0 = qb * B32_ROWS;
  const int m = m0 + tid;
  const bool live = m < S;
  const float* __restrict__ Q = static_cast<const float*>(p.q) + (size_t)bh * S * D;
  const float* __restrict__ dO = static_cast<const float*>(p.dout) + (size_t)bh * S * D;
  const float* __restrict__ K = static_cast<const float*>(p.k) + (size_t)(b * p.Hkv + g) * S * D;
  const float* __restrict__ V = static_cast<const float*>(p.v) + (size_t)(b * p.Hkv + g) * S * D;

  float q[D], dov[D], dq[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    q[d] = live ? Q[(size_t)m * D + d] : 0.f;
    dov[d] = live ? dO[(size_t)m * D + d] : 0.f;
    dq[d] = 0.f;
  }
  if (ROPE != ROPE_NONE && live) rotate_row_f32<D, ROPE>(q, p.table + (size_t)m * (D / 2));
  const float l2 = live ? p.lse2[(size_t)bh * S + m] : INFINITY;
  const float dl = live ? p.delta[(size_t)bh * S + m] : 0.f;

  const float c2 = p.scale * kLog2e;
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;
  const int W = p.window;
  const int ntiles = (S + B32_BT - 1) / B32_BT;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_end = min(ntiles, (min(m0 + B32_ROWS, S) - 1) / B32_BT + 1);
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_begin = max(0, m0 - W + 1) / B32_BT;

  for (int t = t_begin; t < t_end; ++t) {
    const int n0 = t * B32_BT;
    __syncthreads();
    for (int r = 0; r < B32_BT; ++r) {
      const int n = n0 + r;
      for (int d = tid; d < D; d += B32_ROWS) {
        Kf[r][d] = (n < S) ? K[(size_t)n * D + d] : 0.f;
        Vf[r][d] = (n < S) ? V[(size_t)n * D + d] : 0.f;
      }
    }
    __syncthreads();
    if (ROPE != ROPE_NONE && tid < B32_BT && n0 + tid < S) {
      float row[D];
#pragma unroll
      for (int d = 0; d < D; ++d) row[d] = Kf[tid][d];
      rotate_row_f32<D, ROPE>(row, p.table + (size_t)(n0 + tid) * (D / 2));
#pragma unroll
      for (int d = 0; d < D; ++d) Kf[tid][d] = row[d];
    }
    __syncthreads();
    if (!live) continue;
    for (int j = 0; j < B32_BT; ++j) {
      const int n = n0 + j;
      bool ok = n < S;
      if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
      if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
      if (!ok) continue;
      float s = 0.f, dp = 0.f;
#pragma unroll
      for (int d = 0; d < D; ++d) {
        s = __builtin_fmaf(q[d], Kf[j][d], s);
        dp = __builtin_fmaf(dov[d], Vf[j][d], dp);
      }
      const float x = ALIBI ? __builtin_fmaf(s, c2, slope2 * (float)(n - m)) : s * c2;
      const float pr = exp2f(x - l2);
      const float ds = pr * (dp - dl);
#pragma unroll
      for (int d = 0; d < D; ++d) dq[d] = __builtin_fmaf(ds, Kf[j][d], dq[d]);
    }
  }
  if (!live) return;
#pragma unroll
  for (int d = 0; d < D; ++d) dq[d] *= p.scale;
  if (ROPE != ROPE_NONE) rotate_row_f32<D, ROPE, true>(dq, p.table + (size_t)m * (D / 2));
  float* dQ = static_cast<float*>(p.dq) + ((size_t)bh * S + m) * D;
#pragma unroll
  for (int d = 0; d < D; ++d) dQ[d] = dq[d];
}

// One key row per thread (of one batch and K/V head): loops over the group's
// query heads and their visible query tiles, each staged in LDS with Q rotated
// by the first B32_BT threads, dO, and the rows' statistics.
template <int D, int ROPE, int MASK, bool ALIBI>
__global__ __launch_bounds__(64) void bwd_fp32_dkdv_kernel(BwdParams p) {
  __shared__ float Qf[B32_BT][D + 1];
  __shared__ float Of[B32_BT][D + 1];
  __shared__ float Lf[B32_BT], Df[B32_BT];
  const int tid = threadIdx.x;
  const int S = p.S;
  const int BG = p.B * p.Hkv;
  const int bg = blockIdx.x % BG;
  const int kb = (int)(blockIdx.x / BG);
  const int b = bg / p.Hkv, g = bg % p.Hkv;
  const int G = p.H / p.Hkv;
  const int n0 = kb * B32_ROWS;
  const int n = n0 + tid;
  const bool live = n < S;
  const float* __restrict__ K = static_cast<const float*>(p.k) + (size_t)bg * S * D;
  const float* __restrict__ V = static_cast<const float*>(p.v) + (size_t)bg * S * D;

  float k[D], vv[D], dk[D], dv[D];
#pragma unroll
  for (int d = 0; d < D; ++d) {
    k[d] = live ? K[(size_t)n * D + d] : 0.f;
    vv[d] = live ? V[(size_t)n * D + d] : 0.f;
    dk[d] = 0.f;
    dv[d] = 0.f;
  }
  if (ROPE != ROPE_NONE && live) rotate_row_f32<D, ROPE>(k, p.table + (size_t)n * (D / 2));

  const float c2 = p.scale * kLog2e;
  const int W = p.window;
  const int ntiles = (S + B32_BT - 1) / B32_BT;
  const int n_last = min(n0 + B32_ROWS, S) - 1;
  int t_begin = 0, t_end = ntiles;
  if constexpr (MASK != MASK_NONE) t_begin = n0 / B32_BT;
  if constexpr (MASK == MASK_SLIDING_WINDOW) t_end = min(ntiles, (n_last + W - 1) / B32_BT + 1);

  for (int hh = 0; hh < G; ++hh) {
    const int h = g * G + hh;
    const size_t bh = (size_t)b * p.H + h;
    const float* __restrict__ Q = static_cast<const float*>(p.q) + bh * S * D;
    const float* __restrict__ dO = static_cast<const float*>(p.dout) + bh * S * D;
    const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;
    for (int t = t_begin; t < t_end; ++t) {
      const int m0 = t * B32_BT;
      __syncthreads();
      for (int r = 0; r < B32_BT; ++r) {
        const int m = m0 + r;
        for (int d = tid; d < D; d += B32_ROWS) {
          Qf[r][d] = (m < S) ? Q[(size_t)m * D + d] : 0.f;
          Of[r][d] = (m < S) ? dO[(size_t)m * D + d] : 0.f;
        }
      }
      if (tid < B32_BT) {
        const int m = m0 + tid;
        Lf[tid] = (m < S) ? p.lse2[bh * S + m] : INFINITY;
        Df[tid] = (m < S) ? p.delta[bh * S + m] : 0.f;
      }
      __syncthreads();
      if (ROPE != ROPE_NONE && tid < B32_BT && m0 + tid < S) {
        float row[D];
#pragma unroll
        for (int d = 0; d < D; ++d) row[d] = Qf[tid][d];
        rotate_row_f32<D, ROPE>(row, p.table + (size_t)(m0 + tid) * (D / 2));
#pragma unroll
        for (int d = 0; d < D; ++d) Qf[tid][d] = row[d];
      }
      __syncthreads();
      if (!live) continue;
      for (int i = 0; i < B32_BT; ++i) {
        const int m = m0 + i;
        bool ok = m < S;
        if constexpr (MASK != MASK_NONE) ok = ok && (n <= m);
        if constexpr (MASK == MASK_SLIDING_WINDOW) ok = ok && (n > m - W);
        if (!ok) continue;
        float s = 0.f, dp = 0.f;
#pragma unroll
        for (int d = 0; d < D; ++d) {
          s = __builtin_fmaf(k[d], Qf[i][d], s);
          dp = __builtin_fmaf(vv[d], Of[i][d], dp);
        }
        const float x = ALIBI ? __builtin_fmaf(s, c2, slope2 * (float)(n - m)) : s * c2;
        const float pr = exp2f(x - Lf[i]);
        const float ds = pr * (dp - Df[i]);
#pragma unroll
        for (int d = 0; d < D; ++d) {
          dv[d] = __builtin_fmaf(pr, Of[i][d], dv[d]);
          dk[d] = __builtin_fmaf(ds, Qf[i][d], dk[d]);
        }
      }
    }
  }
  if (!live) return;
#pragma unroll
  for (int d = 0; d < D; ++d) dk[d] *= p.scale;
  if (ROPE != ROPE_NONE) rotate_row_f32<D, ROPE, true>(dk, p.table + (size_t)n * (D / 2));
  float* dK = static_cast<float*>(p.dk) + ((size_t)bg * S + n) * D;
  float* dV = static_cast<float*>(p.dv) + ((size_t)bg * S + n) * D;
#pragma unroll
  for (int d = 0; d < D; ++d) {
    dK[d] = dk[d];
    dV[d] = dv[d];
  }
}

template <int D, int ROPE, int MASK, bool ALIBI>
static int launch_one(const BwdParams& p, hipStream_t st) {
  const long long rows = (long long)p.B * p.H * p.S;
  hipLaunchKernelGGL(bwd_fp32_prep_kernel, dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, st, p, D);
  const int nb = (p.S + B32_ROWS - 1) / B32_ROWS;
  hipLaunchKernelGGL((bwd_fp32_dkdv_kernel<D, ROPE, MASK, ALIBI>), dim3((unsigned)(nb * p.B * p.Hkv)), dim3(B32_ROWS),
                     0, st, p);
  hipLaunchKernelGGL((bwd_fp32_dq_kernel<D, ROPE, MASK, ALIBI>), dim3((unsigned)(nb * p.B * p.H)), dim3(B32_ROWS), 0,
                     st, p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

template <int D, int ROPE>
static int dispatch_mask(int mask, bool alibi, const BwdParams& p, hipStream_t st) {
  switch (mask) {
    case MASK_NONE: return alibi ? launch_one<D, ROPE, MASK_NONE, true>(p, st) : launch_one<D, ROPE, MASK_NONE, false>(p, st);
    case MASK_CAUSAL: return alibi ? launch_one<D, ROPE, MASK_CAUSAL, true>(p, st) : launch_one<D, ROPE, MASK_CAUSAL, false>(p, st);
    case MASK_SLIDING_WINDOW: return alibi ? launch_one<D, ROPE, MASK_SLIDING_WINDOW, true>(p, st) : launch_one<D, ROPE, MASK_SLIDING_WINDOW, false>(p, st);
  }
  return -2;
}

template <int D>
static int dispatch_rope(int rope, int mask, bool alibi, const BwdParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return dispatch_mask<D, ROPE_NONE>(mask, alibi, p, st);
    case ROPE_NEOX: return dispatch_mask<D, ROPE_NEOX>(mask, alibi, p, st);
    case ROPE_INTERLEAVED: return dispatch_mask<D, ROPE_INTERLEAVED>(mask, alibi, p, st);
  }
  return -2;
}

int launch_bwd_fp32(int D, int rope, int mask, bool alibi, const BwdParams& p, hipStream_t st) {
  if (D == 64) return dispatch_rope<64>(rope, mask, alibi, p, st);
  if (D == 128) return dispatch_rope<128>(rope, mask, alibi, p, st);
  return -2;
}

}  // namespace af
