// C-ABI entry points (declared in include/attnfuse.h): argument validation,
// the per-device cos/sin table cache, and dispatch to the kernel launchers.
// Every argument is checked before the first HIP call; no exception leaves
// this file.
#include "attnfuse.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <vector>

#include "launch.hpp"

namespace {

constexpr int kMaxS = 1 << 20;
constexpr int kAbiVersion = 2;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// Block-sparse masks: 64-position blocks, at most 2048 per side (the per-
// workgroup tile list lives in LDS).
constexpr int kMaxSparseS = 64 * 2048;


int map_launch(int rc) {
  if (rc == 0) return AF_OK;
  if (rc == -2) return AF_ERR_UNSUPPORTED;
  return AF_ERR_HIP;
}

// ---------------------------------------------------------------- cos/sin table cache
struct RopeTable {
  int device;
  int D;
  uint32_t theta_bits;
  int rows;
  float2* ptr;
};
std::mutex g_table_mu;
std::vector<RopeTable> g_tables;   // never freed: kernels on any stream may still read them

int rope_table(int D, float theta, int S, hipStream_t stream, const float2** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return AF_ERR_HIP;
  uint32_t bits;
  std::memcpy(&bits, &theta, sizeof bits);
  std::lock_guard<std::mutex> lock(g_table_mu);
  for (const RopeTable& t : g_tables) {
    if (t.device == dev && t.D == D && t.theta_bits == bits && t.rows >= S) {
      *out = t.ptr;
      return AF_OK;
    }
  }
  int rows = 4096;
  while (rows < S) rows *= 2;
  float2* ptr = nullptr;
  if (hipMalloc(&ptr, (size_t)rows * (D / 2) * sizeof(float2)) != hipSuccess) return AF_ERR_HIP;
  if (af::launch_rope_table(ptr, rows, D, (double)theta, stream) != 0 || hipStreamSynchronize(stream) != hipSuccess) {
    (void)hipFree(ptr);
    return AF_ERR_HIP;
  }
  g_tables.push_back({dev, D, bits, rows, ptr});
  *out = ptr;
  return AF_OK;
}

// ---------------------------------------------------------------- validation
int check_common(int B, int H, int H_kv, int S, int D, int dtype, int rope, float rope_theta) {
  if (B < 1 || H < 1 || H_kv < 1 || S < 1 || S > kMaxS || D < 2 || (D & 1)) return AF_ERR_INVALID_ARG;
  if (H % H_kv != 0) return AF_ERR_INVALID_ARG;
  if (dtype != AF_DTYPE_BF16 && dtype != AF_DTYPE_FP32) return AF_ERR_INVALID_ARG;
  if (rope != AF_ROPE_NONE && rope != AF_ROPE_NEOX && rope != AF_ROPE_INTERLEAVED) return AF_ERR_INVALID_ARG;
  if (rope != AF_ROPE_NONE && !(std::isfinite(rope_theta) && rope_theta > 0.f)) return AF_ERR_INVALID_ARG;
  // grid sizes and element offsets must stay inside their integer types
  if ((long long)B * H * ((S + 63) / 64) >= (1LL << 31)) return AF_ERR_INVALID_ARG;
  return AF_OK;
}

int check_attn(int mask, int window, float scale) {
  if (mask != AF_MASK_NONE && mask != AF_MASK_CAUSAL && mask != AF_MASK_SLIDING_WINDOW) return AF_ERR_INVALID_ARG;
  if (mask == AF_MASK_SLIDING_WINDOW && window < 1) return AF_ERR_INVALID_ARG;
  if (!(std::isfinite(scale) && scale > 0.f)) return AF_ERR_INVALID_ARG;
  return AF_OK;
}

bool supported_d(int D) { return D == 64 || D == 128; }

// Backward workspace: [delta f32 | lse2 f32 | dO fp16 | Q' fp16 | K' fp16], each
// section starting on a 256-byte boundary; the last two only with RoPE.
struct BwdWorkspace {
  size_t delta, lse2, do16, qr16, kr16, total;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

BwdWorkspace bwd_workspace(int B, int H, int H_kv, int S, int D, int rope) {
  const size_t rows = (size_t)B * H * S, krows = (size_t)B * H_kv * S;
  BwdWorkspace w{};
  size_t off = 0;
  w.delta = off; off += align256(rows * sizeof(float));
  w.lse2 = off;  off += align256(rows * sizeof(float));
  w.do16 = off;  off += align256(rows * D * 2);
  if (rope != AF_ROPE_NONE) {
    w.qr16 = off; off += align256(rows * D * 2);
    w.kr16 = off; off += align256(krows * D * 2);
  }
  w.total = off;
  return w;
}

// Decode workspace: per-wave partial (max, sum) pairs, then accumulators
// (four phase-1 waves per chunk, each writing its own partial).
struct DecodeLayout {
  int chunk, nsplit;
  size_t ml, acc, total;
};

// Keys per phase-1 workgroup: a power of two in [128, 4096] giving about 512
// workgroups (one resident round at two per CU, so each wave streams several
// tiles); the wave partials' (max, sum) pairs then accumulators, each
// 256-byte aligned.
DecodeLayout decode_layout(int B, int H, int H_kv, int S, int D) {
  const long long work = (long long)B * H_kv * S;
  DecodeLayout L{};
  L.chunk = 128;
  while (L.chunk < 4096 && (long long)L.chunk * 512 < work) L.chunk *= 2;
  L.nsplit = (S + L.chunk - 1) / L.chunk;
  const size_t parts = (size_t)B * H * L.nsplit * 4;
  L.ml = 0;
  L.acc = align256(parts * 2 * sizeof(float));
  L.total = L.acc + align256(parts * D * sizeof(float));
  return L;
}

// ---------------------------------------------------------------- shared bodies
// Dense bias tensor and normalisation of the extended entry points (EXT_NONE
// for the plain ones).
struct Ext {
  const float* bias = nullptr;
  long long sb = 0, sh = 0, sq = 0;
  int norm = AF_NORM_SOFTMAX;
  int kind() const {
    if (norm == AF_NORM_RELU) return bias ? af::EXT_RELU_BIAS : af::EXT_RELU;
    return bias ? af::EXT_BIAS : af::EXT_NONE;
  }
};

int check_ext(const Ext& e, const void* const* outs, int nouts) {
  if (e.norm != AF_NORM_SOFTMAX && e.norm != AF_NORM_RELU) return AF_ERR_INVALID_ARG;
  if (e.bias) {
    if ((reinterpret_cast<uintptr_t>(e.bias) & 3u) != 0) return AF_ERR_INVALID_ARG;
    if (e.sb < 0 || e.sh < 0 || e.sq < 0) return AF_ERR_INVALID_ARG;
    for (int i = 0; i < nouts; ++i) if (outs[i] == (const void*)e.bias) return AF_ERR_INVALID_ARG;
  }
  return AF_OK;
}

int fwd_impl(const void* Q, const void* K, const void* V, void* O, float* LSE, const int* q_block_ptr,
             const int* k_block_idx, const Ext& ext, int B, int H, int H_kv, int S, int D, int dtype, int rope,
             float rope_theta, int mask, int window, const float* alibi_slopes, float softmax_scale, void* stream) {
  const bool relu = ext.norm == AF_NORM_RELU;   // no row statistic: LSE may be NULL
  if (!Q || !K || !V || !O || (!LSE && !relu)) return AF_ERR_INVALID_ARG;
  if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O) || !aligned16(LSE)) return AF_ERR_INVALID_ARG;
  if (O == Q || O == K || O == V || (const void*)LSE == Q || (const void*)LSE == K || (const void*)LSE == V)
    return AF_ERR_INVALID_ARG;
  const void* outs[] = {O, LSE};
  int rc0 = check_ext(ext, outs, 2);
  if (rc0 != AF_OK) return rc0;
  int rc = check_common(B, H, H_kv, S, D, dtype, rope, rope_theta);
  if (rc != AF_OK) return rc;
  if ((rc = check_attn(mask, window, softmax_scale)) != AF_OK) return rc;
  if (!supported_d(D)) return AF_ERR_UNSUPPORTED;
  if (q_block_ptr && dtype == AF_DTYPE_FP32) return AF_ERR_UNSUPPORTED;   // block-sparse: bf16 kernels only
  // the bias tensor and relu attention: bf16, without ALiBi or a block mask
  if (ext.kind() != af::EXT_NONE && (dtype == AF_DTYPE_FP32 || alibi_slopes || q_block_ptr))
    return AF_ERR_UNSUPPORTED;

  hipStream_t st = static_cast<hipStream_t>(stream);
  af::FwdParams p{};
  p.q = Q; p.k = K; p.v = V; p.o = O; p.lse = LSE;
  p.B = B; p.H = H; p.Hkv = H_kv; p.S = S;
  // a window of S or more keys is the causal mask; clamping keeps n + window in int range
  p.window = (mask == AF_MASK_SLIDING_WINDOW) ? (window < S ? window : S) : 0;
  p.slopes = alibi_slopes;
  p.scale = softmax_scale;
  p.table = nullptr;
  p.bq_ptr = q_block_ptr;
  p.bk_idx = k_block_idx;
  p.bias = ext.bias;
  p.bias_sb = ext.sb; p.bias_sh = ext.sh; p.bias_sq = ext.sq;
  if (rope != AF_ROPE_NONE && (rc = rope_table(D, rope_theta, S, st, &p.table)) != AF_OK) return rc;
  const bool alibi = alibi_slopes != nullptr;
  if (dtype == AF_DTYPE_BF16) return map_launch(af::launch_fwd_bf16(D, rope, mask, alibi, ext.kind(), p, st));
  return map_launch(af::launch_fwd_fp32(D, rope, mask, alibi, p, st));
}

// sparse: NULL (dense) or {q_block_ptr, k_block_idx, k_block_ptr, q_block_idx}
int bwd_impl(const void* Q, const void* K, const void* V, const void* O, const void* dO, const float* LSE, void* dQ,
             void* dK, void* dV, const int* const* sparse, const Ext& ext, void* workspace, size_t workspace_bytes,
             int B, int H, int H_kv, int S, int D, int dtype, int rope, float rope_theta, int mask, int window,
             const float* alibi_slopes, float softmax_scale, void* stream) {
  const bool relu = ext.norm == AF_NORM_RELU;   // the LSE is not used: it may be NULL
  if (relu) LSE = nullptr;
  const void* ins[] = {Q, K, V, O, dO, LSE};
  void* outs[] = {dQ, dK, dV, workspace};
  for (const void* x : ins) if (!aligned16(x)) return AF_ERR_INVALID_ARG;
  if (!Q || !K || !V || !O || !dO || (!LSE && !relu)) return AF_ERR_INVALID_ARG;
  for (const void* x : outs) if (!x || !aligned16(x)) return AF_ERR_INVALID_ARG;
  for (const void* x : outs)
    for (const void* y : ins) if (y && x == y) return AF_ERR_INVALID_ARG;
  int rc0 = check_ext(ext, outs, 4);
  if (rc0 != AF_OK) return rc0;
  int rc = check_common(B, H, H_kv, S, D, dtype, rope, rope_theta);
  if (rc != AF_OK) return rc;
  if ((rc = check_attn(mask, window, softmax_scale)) != AF_OK) return rc;
  if (workspace_bytes < attnfuse_bwd_workspace_bytes(B, H, H_kv, S, D, rope)) return AF_ERR_INVALID_ARG;
  if (!supported_d(D)) return AF_ERR_UNSUPPORTED;
  if (sparse && dtype == AF_DTYPE_FP32) return AF_ERR_UNSUPPORTED;        // block-sparse: bf16 kernels only
  if (ext.kind() != af::EXT_NONE && (dtype == AF_DTYPE_FP32 || alibi_slopes || sparse)) return AF_ERR_UNSUPPORTED;

  hipStream_t st = static_cast<hipStream_t>(stream);
  af::BwdParams p{};
  p.q = Q; p.k = K; p.v = V; p.o = O; p.dout = dO; p.lse = LSE;
  p.dq = dQ; p.dk = dK; p.dv = dV;
  const BwdWorkspace ws = bwd_workspace(B, H, H_kv, S, D, rope);
  char* wb = static_cast<char*>(workspace);
  p.delta = reinterpret_cast<float*>(wb + ws.delta);
  p.lse2 = reinterpret_cast<float*>(wb + ws.lse2);
  p.do16 = wb + ws.do16;
  p.qr16 = (rope != AF_ROPE_NONE) ? wb + ws.qr16 : nullptr;
  p.kr16 = (rope != AF_ROPE_NONE) ? wb + ws.kr16 : nullptr;
  p.B = B; p.H = H; p.Hkv = H_kv; p.S = S;
  // a window of S or more keys is the causal mask; clamping keeps n + window in int range
  p.window = (mask == AF_MASK_SLIDING_WINDOW) ? (window < S ? window : S) : 0;
  p.slopes = alibi_slopes;
  p.scale = softmax_scale;
  p.table = nullptr;
  if (sparse) {
    p.bq_ptr = sparse[0]; p.bk_idx = sparse[1];
    p.bk_ptr = sparse[2]; p.bq_idx = sparse[3];
  }
  p.bias = ext.bias;
  p.bias_sb = ext.sb; p.bias_sh = ext.sh; p.bias_sq = ext.sq;
  if (rope != AF_ROPE_NONE && (rc = rope_table(D, rope_theta, S, st, &p.table)) != AF_OK) return rc;
  const bool alibi = alibi_slopes != nullptr;
  if (dtype == AF_DTYPE_FP32) return map_launch(af::launch_bwd_fp32(D, rope, mask, alibi, p, st));
  return map_launch(af::launch_bwd_bf16(D, rope, mask, alibi, ext.kind(), p, st));
}

}  // namespace

extern "C" {

int attnfuse_version(void) { return kAbiVersion; }

const char* attnfuse_strerror(int code) {
  switch (code) {
    case AF_OK: return "success";
    case AF_ERR_INVALID_ARG: return "invalid argument";
    case AF_ERR_UNSUPPORTED: return "unsupported variant (no compiled kernel)";
    case AF_ERR_HIP: return "HIP runtime error";
  }
  return "unknown error code";
}

int attnfuse_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE,
                 int B, int H, int H_kv, int S, int D, int dtype,
                 int rope, float rope_theta, int mask, int window,
                 const float* alibi_slopes, float softmax_scale, void* stream) {
  return fwd_impl(Q, K, V, O, LSE, nullptr, nullptr, Ext{}, B, H, H_kv, S, D, dtype, rope, rope_theta, mask, window,
                  alibi_slopes, softmax_scale, stream);
}

int attnfuse_fwd_blocksparse(const void* Q, const void* K, const void* V, void* O, float* LSE,
                             const int* q_block_ptr, const int* k_block_idx,
                             int B, int H, int H_kv, int S, int D, int dtype,
                             int rope, float rope_theta, int mask, int window,
                             const float* alibi_slopes, float softmax_scale, void* stream) {
  if (!q_block_ptr || !k_block_idx || !aligned4(q_block_ptr) || !aligned4(k_block_idx)) return AF_ERR_INVALID_ARG;
  const void* outs[] = {O, LSE};
  for (const void* x : outs)
    if (x == (const void*)q_block_ptr || x == (const void*)k_block_idx) return AF_ERR_INVALID_ARG;
  if (S < 1 || S > kMaxSparseS) return AF_ERR_INVALID_ARG;
  return fwd_impl(Q, K, V, O, LSE, q_block_ptr, k_block_idx, Ext{}, B, H, H_kv, S, D, dtype, rope, rope_theta, mask,
                  window, alibi_slopes, softmax_scale, stream);
}

int attnfuse_fwd_bias_norm(const void* Q, const void* K, const void* V, void* O, float* LSE,
                           const float* bias, long long bias_stride_b, long long bias_stride_h,
                           long long bias_stride_q, int norm,
                           int B, int H, int H_kv, int S, int D, int dtype,
                           int rope, float rope_theta, int mask, int window,
                           const float* alibi_slopes, float softmax_scale, void* stream) {
  Ext e;
  e.bias = bias; e.sb = bias_stride_b; e.sh = bias_stride_h; e.sq = bias_stride_q; e.norm = norm;
  return fwd_impl(Q, K, V, O, LSE, nullptr, nullptr, e, B, H, H_kv, S, D, dtype, rope, rope_theta, mask, window,
                  alibi_slopes, softmax_scale, stream);
}

size_t attnfuse_bwd_workspace_bytes(int B, int H, int H_kv, int S, int D, int rope) {
  if (B < 1 || H < 1 || H_kv < 1 || S < 1 || D < 2 || (D & 1)) return 0;
  if (rope != AF_ROPE_NONE && rope != AF_ROPE_NEOX && rope != AF_ROPE_INTERLEAVED) return 0;
  return bwd_workspace(B, H, H_kv, S, D, rope).total;
}

int attnfuse_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int H_kv, int S, int D, int dtype,
                 int rope, float rope_theta, int mask, int window,
                 const float* alibi_slopes, float softmax_scale, void* stream) {
  return bwd_impl(Q, K, V, O, dO, LSE, dQ, dK, dV, nullptr, Ext{}, workspace, workspace_bytes, B, H, H_kv, S, D,
                  dtype, rope, rope_theta, mask, window, alibi_slopes, softmax_scale, stream);
}

int attnfuse_bwd_blocksparse(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                             const float* LSE, void* dQ, void* dK, void* dV,
                             const int* q_block_ptr, const int* k_block_idx,
                             const int* k_block_ptr, const int* q_block_idx,
                             void* workspace, size_t workspace_bytes,
                             int B, int H, int H_kv, int S, int D, int dtype,
                             int rope, float rope_theta, int mask, int window,
                             const float* alibi_slopes, float softmax_scale, void* stream) {
  const int* m[] = {q_block_ptr, k_block_idx, k_block_ptr, q_block_idx};
  for (const int* x : m) if (!x || !aligned4(x)) return AF_ERR_INVALID_ARG;
  const void* outs[] = {dQ, dK, dV, workspace};
  for (const void* x : outs)
    for (const int* y : m) if (x == (const void*)y) return AF_ERR_INVALID_ARG;
  if (S < 1 || S > kMaxSparseS) return AF_ERR_INVALID_ARG;
  return bwd_impl(Q, K, V, O, dO, LSE, dQ, dK, dV, m, Ext{}, workspace, workspace_bytes, B, H, H_kv, S, D, dtype,
                  rope, rope_theta, mask, window, alibi_slopes, softmax_scale, stream);
}

int attnfuse_bwd_bias_norm(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                           const float* LSE, void* dQ, void* dK, void* dV,
                           const float* bias, long long bias_stride_b, long long bias_stride_h,
                           long long bias_stride_q, int norm,
                           void* workspace, size_t workspace_bytes,
                           int B, int H, int H_kv, int S, int D, int dtype,
                           int rope, float rope_theta, int mask, int window,
                           const float* alibi_slopes, float softmax_scale, void* stream) {
  Ext e;
  e.bias = bias; e.sb = bias_stride_b; e.sh = bias_stride_h; e.sq = bias_stride_q; e.norm = norm;
  return bwd_impl(Q, K, V, O, dO, LSE, dQ, dK, dV, nullptr, e, workspace, workspace_bytes, B, H, H_kv, S, D, dtype,
                  rope, rope_theta, mask, window, alibi_slopes, softmax_scale, stream);
}

// ---------------------------------------------------------------- decode
size_t attnfuse_decode_workspace_bytes(int B, int H, int H_kv, int S_kv, int D) {
  if (B < 1 || H < 1 || H_kv < 1 || S_kv < 1 || S_kv > kMaxS || D < 2 || (D & 1) || H % H_kv) return 0;
  return decode_layout(B, H, H_kv, S_kv, D).total;
}

int attnfuse_decode(const void* Q, const void* K, const void* V, const int* cache_lens,
                    void* O, float* LSE, void* workspace, size_t workspace_bytes,
                    int B, int H, int H_kv, int S_kv, int D, int dtype,
                    int rope, float rope_theta, int mask, int window,
                    const float* alibi_slopes, float softmax_scale, void* stream) {
  const void* ins[] = {Q, K, V};
  const void* outs[] = {O, LSE, workspace};
  for (const void* x : ins) if (!x || !aligned16(x)) return AF_ERR_INVALID_ARG;
  for (const void* x : outs) if (!x || !aligned16(x)) return AF_ERR_INVALID_ARG;
  if (cache_lens && (reinterpret_cast<uintptr_t>(cache_lens) & 3u)) return AF_ERR_INVALID_ARG;
  for (const void* x : outs) {
    for (const void* y : ins) if (x == y) return AF_ERR_INVALID_ARG;
    if (x == static_cast<const void*>(cache_lens)) return AF_ERR_INVALID_ARG;
  }
  int rc = check_common(B, H, H_kv, S_kv, D, dtype, rope, rope_theta);
  if (rc != AF_OK) return rc;
  if ((rc = check_attn(mask, window, softmax_scale)) != AF_OK) return rc;
  if (workspace_bytes < attnfuse_decode_workspace_bytes(B, H, H_kv, S_kv, D)) return AF_ERR_INVALID_ARG;
  if (!supported_d(D) || dtype != AF_DTYPE_BF16 || H / H_kv > 32) return AF_ERR_UNSUPPORTED;

  hipStream_t st = static_cast<hipStream_t>(stream);
  const DecodeLayout L = decode_layout(B, H, H_kv, S_kv, D);
  af::DecodeParams p{};
  p.q = Q; p.k = K; p.v = V; p.lens = cache_lens; p.o = O; p.lse = LSE;
  char* wb = static_cast<char*>(workspace);
  p.part_ml = reinterpret_cast<float*>(wb + L.ml);
  p.part_acc = reinterpret_cast<float*>(wb + L.acc);
  p.B = B; p.H = H; p.Hkv = H_kv; p.S = S_kv;
  p.window = (mask == AF_MASK_SLIDING_WINDOW) ? (window < S_kv ? window : S_kv) : 0;
  p.chunk = L.chunk; p.nsplit = L.nsplit;
  p.slopes = alibi_slopes;
  p.scale = softmax_scale;
  p.table = nullptr;
  if (rope != AF_ROPE_NONE && (rc = rope_table(D, rope_theta, S_kv, st, &p.table)) != AF_OK) return rc;
  return map_launch(af::launch_decode(D, rope, alibi_slopes != nullptr, p, st));
}

static int rope_common(const void* X0, const void* X1, void* Y0, void* Y1, int B, int H, int H_kv, int S, int D,
                       int dtype, int rope, float rope_theta, void* stream, bool inverse) {
  if (!X0 || !Y0 || !aligned16(X0) || !aligned16(Y0)) return AF_ERR_INVALID_ARG;
  if ((X1 == nullptr) != (Y1 == nullptr)) return AF_ERR_INVALID_ARG;
  if (X1 && (!aligned16(X1) || !aligned16(Y1))) return AF_ERR_INVALID_ARG;
  if (!X1) H_kv = 1;
  int rc = check_common(B, H, H_kv, S, D, dtype, rope, rope_theta);
  if (rc != AF_OK) return rc;
  if (rope == AF_ROPE_NONE) return AF_ERR_INVALID_ARG;
  if (!supported_d(D)) return AF_ERR_UNSUPPORTED;
  hipStream_t st = static_cast<hipStream_t>(stream);
  af::RopeParams p{};
  p.x0 = X0; p.y0 = Y0; p.heads0 = H;
  p.x1 = X1; p.y1 = Y1; p.heads1 = X1 ? H_kv : 0;
  p.B = B; p.S = S;
  if ((rc = rope_table(D, rope_theta, S, st, &p.table)) != AF_OK) return rc;
  return map_launch(af::launch_rope(dtype == AF_DTYPE_FP32, D, rope, inverse, p, st));
}

int attnfuse_rope(const void* Q, const void* K, void* Qr, void* Kr, int B, int H, int H_kv, int S, int D,
                  int dtype, int rope, float rope_theta, void* stream) {
  return rope_common(Q, K, Qr, Kr, B, H, H_kv, S, D, dtype, rope, rope_theta, stream, false);
}

int attnfuse_rope_bwd(const void* dQr, const void* dKr, void* dQ, void* dK, int B, int H, int H_kv, int S, int D,
                      int dtype, int rope, float rope_theta, void* stream) {
  return rope_common(dQr, dKr, dQ, dK, B, H, H_kv, S, D, dtype, rope, rope_theta, stream, true);
}

}  // extern "C"
