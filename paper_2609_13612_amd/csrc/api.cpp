// C-ABI entry points (declared in include/attnfuse.h): argument validation
// and dispatch to the kernel launchers.  Every argument is checked before the
// first HIP call; no exception leaves this file.  Nothing here allocates,
// synchronises or keeps state: the caller owns every buffer, the RoPE table
// included.
#include "attnfuse.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>

#include "launch.hpp"

namespace {

constexpr int kMaxS = 1 << 20;
static_assert(AF_DECODE_SCRATCH_BYTES == af::DECODE_SCRATCH_BYTES, "header and library agree on the static scratch");
constexpr int kAbiVersion = 3;

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

// ---------------------------------------------------------------- caller-owned cos/sin table
// The table is [rows][D/2] (cos, sin) fp32 pairs; a RoPE call reads rows 0..S-1.
constexpr int kMaxTableRows = kMaxS;

size_t table_bytes(int rows, int D) { return (size_t)rows * (size_t)(D / 2) * 2 * sizeof(float); }

// Checks the table arguments of a call that rotates positions 0..S-1 (nothing
// without RoPE); a table given as an output would be a caller error too.
int check_table(int rope, const float* table, int rows, int S, const void* const* outs, int nouts) {
  if (rope == AF_ROPE_NONE) return AF_OK;
  if (!table || !aligned16(table) || rows < S || rows > kMaxTableRows) return AF_ERR_INVALID_ARG;
  for (int i = 0; i < nouts; ++i)
    if (outs[i] == static_cast<const void*>(table)) return AF_ERR_INVALID_ARG;
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

// Backward workspace: [delta f32 | lse2 f32 | dO fp16 | dO scale f32 | partial
// max |dO| u32 | Q' fp16 | K' fp16], each section starting on a 256-byte
// boundary; the last two only with RoPE.  The partial maxima cover chunks of
// kDmaxChunk elements of each (batch, K/V head)'s dO.
constexpr long long kDmaxChunk = 16384;

struct BwdWorkspace {
  size_t delta, lse2, do16, dscale, dmax, qr16, kr16, total;
  int dmax_chunks;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

BwdWorkspace bwd_workspace(int B, int H, int H_kv, int S, int D, int rope) {
  const size_t rows = (size_t)B * H * S, krows = (size_t)B * H_kv * S;
  BwdWorkspace w{};
  size_t off = 0;
  w.delta = off; off += align256(rows * sizeof(float));
  w.lse2 = off;  off += align256(rows * sizeof(float));
  w.do16 = off;  off += align256(rows * D * 2);
  const size_t groups = (size_t)B * H_kv;
  w.dmax_chunks = (int)(((long long)(H / H_kv) * S * D + kDmaxChunk - 1) / kDmaxChunk);
  w.dscale = off; off += align256(groups * sizeof(float));
  w.dmax = off;   off += align256(groups * w.dmax_chunks * sizeof(uint32_t));
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
             float rope_theta, const float* rope_table, int rope_table_rows, int mask, int window,
             const float* alibi_slopes, float softmax_scale, void* stream) {
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
  if ((rc = check_table(rope, rope_table, rope_table_rows, S, outs, 2)) != AF_OK) return rc;
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
  p.table = (rope != AF_ROPE_NONE) ? reinterpret_cast<const float2*>(rope_table) : nullptr;
  p.bq_ptr = q_block_ptr;
  p.bk_idx = k_block_idx;
  p.bias = ext.bias;
  p.bias_sb = ext.sb; p.bias_sh = ext.sh; p.bias_sq = ext.sq;
  const bool alibi = alibi_slopes != nullptr;
  if (dtype == AF_DTYPE_BF16) return map_launch(af::launch_fwd_bf16(D, rope, mask, alibi, ext.kind(), p, st));
  return map_launch(af::launch_fwd_fp32(D, rope, mask, alibi, p, st));
}

// sparse: NULL (dense) or {q_block_ptr, k_block_idx, k_block_ptr, q_block_idx}
int bwd_impl(const void* Q, const void* K, const void* V, const void* O, const void* dO, const float* LSE, void* dQ,
             void* dK, void* dV, const int* const* sparse, const Ext& ext, void* workspace, size_t workspace_bytes,
             int B, int H, int H_kv, int S, int D, int dtype, int rope, float rope_theta, const float* rope_table,
             int rope_table_rows, int mask, int window, const float* alibi_slopes, float softmax_scale,
             void* stream) {
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
  if ((rc = check_table(rope, rope_table, rope_table_rows, S, outs, 4)) != AF_OK) return rc;
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
  p.dscale = reinterpret_cast<float*>(wb + ws.dscale);
  p.dmax = reinterpret_cast<uint32_t*>(wb + ws.dmax);
  p.dmax_chunks = ws.dmax_chunks;
  p.qr16 = (rope != AF_ROPE_NONE) ? wb + ws.qr16 : nullptr;
  p.kr16 = (rope != AF_ROPE_NONE) ? wb + ws.kr16 : nullptr;
  p.B = B; p.H = H; p.Hkv = H_kv; p.S = S;
  // a window of S or more keys is the causal mask; clamping keeps n + window in int range
  p.window = (mask == AF_MASK_SLIDING_WINDOW) ? (window < S ? window : S) : 0;
  p.slopes = alibi_slopes;
  p.scale = softmax_scale;
  p.table = (rope != AF_ROPE_NONE) ? reinterpret_cast<const float2*>(rope_table) : nullptr;
  if (sparse) {
    p.bq_ptr = sparse[0]; p.bk_idx = sparse[1];
    p.bk_ptr = sparse[2]; p.bq_idx = sparse[3];
  }
  p.bias = ext.bias;
  p.bias_sb = ext.sb; p.bias_sh = ext.sh; p.bias_sq = ext.sq;
  const bool alibi = alibi_slopes != nullptr;
  if (dtype == AF_DTYPE_FP32) return map_launch(af::launch_bwd_fp32(D, rope, mask, alibi, p, st));
  return map_launch(af::launch_bwd_bf16(D, rope, mask, alibi, ext.kind(), p, st));
}

}  // namespace

extern "C" {

int attnfuse_version(void) { return kAbiVersion; }
                     
size_t attnfuse_rope_table_bytes(int rows, int D) {
  if (rows < 1 || rows > kMaxTableRows || D < 2 || (D & 1)) return 0;
  return table_bytes(rows, D);
}

int attnfuse_rope_table_fill(float* table, int rows, int D, float rope_theta, void* stream) {
  if (!table || !aligned16(table) || rows < 1 || rows > kMaxTableRows || D < 2 || (D & 1)) return AF_ERR_INVALID_ARG;
  if (!(std::isfinite(rope_theta) && rope_theta > 0.f)) return AF_ERR_INVALID_ARG;
  if (!supported_d(D)) return AF_ERR_UNSUPPORTED;
  return map_launch(af::launch_rope_table(reinterpret_cast<float2*>(table), rows, D, (double)rope_theta,
                                          static_cast<hipStream_t>(stream)));
}

const char* attnfuse_strerror(int code) {
  switch (code) {
    case AF_OK: return "success";
    case AF_ERR_INVALID_ARG: return "invalid argument";
    case AF_ERR_UNSUPPORTED: return "unsupported variant (no compiled kernel)";
    case AF_ERR_HIP: return "HIP runtime error";
    case AF_ERR_TOO_LARGE: return "request needs more than the library's static scratch (use the workspace entry point)";
  }
  return "unknown error code";
}

int attnfuse_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE,
                 int B, int H, int H_kv, int S, int D, int dtype,
                 int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                 int mask, int window,
                 const float* alibi_slopes, float softmax_scale, void* stream) {
  return fwd_impl(Q, K, V, O, LSE, nullptr, nullptr, Ext{}, B, H, H_kv, S, D, dtype, rope, rope_theta, rope_table,
                  rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream);
}

int attnfuse_fwd_blocksparse(const void* Q, const void* K, const void* V, void* O, float* LSE,
                             const int* q_block_ptr, const int* k_block_idx,
                             int B, int H, int H_kv, int S, int D, int dtype,
                             int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                             int mask, int window,
                             const float* alibi_slopes, float softmax_scale, void* stream) {
  if (!q_block_ptr || !k_block_idx || !aligned4(q_block_ptr) || !aligned4(k_block_idx)) return AF_ERR_INVALID_ARG;
  const void* outs[] = {O, LSE};
  for (const void* x : outs)
    if (x == (const void*)q_block_ptr || x == (const void*)k_block_idx) return AF_ERR_INVALID_ARG;
  if (S < 1 || S > kMaxSparseS) return AF_ERR_INVALID_ARG;
  return fwd_impl(Q, K, V, O, LSE, q_block_ptr, k_block_idx, Ext{}, B, H, H_kv, S, D, dtype, rope, rope_theta,
                  rope_table, rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream);
}

int attnfuse_fwd_bias_norm(const void* Q, const void* K, const void* V, void* O, float* LSE,
                           const float* bias, long long bias_stride_b, long long bias_stride_h,
                           long long bias_stride_q, int norm,
                           int B, int H, int H_kv, int S, int D, int dtype,
                           int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                           int mask, int window,
                           const float* alibi_slopes, float softmax_scale, void* stream) {
  Ext e;
  e.bias = bias; e.sb = bias_stride_b; e.sh = bias_stride_h; e.sq = bias_stride_q; e.norm = norm;
  return fwd_impl(Q, K, V, O, LSE, nullptr, nullptr, e, B, H, H_kv, S, D, dtype, rope, rope_theta, rope_table,
                  rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream);
}

size_t attnfuse_bwd_workspace_bytes(int B, int H, int H_kv, int S, int D, int rope) {
  if (B < 1 || H < 1 || H_kv < 1 || S < 1 || D < 2 || (D & 1) || H % H_kv) return 0;
  if (rope != AF_ROPE_NONE && rope != AF_ROPE_NEOX && rope != AF_ROPE_INTERLEAVED) return 0;
  return bwd_workspace(B, H, H_kv, S, D, rope).total;
}

int attnfuse_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int H_kv, int S, int D, int dtype,
                 int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                 int mask, int window,
                 const float* alibi_slopes, float softmax_scale, void* stream) {
  return bwd_impl(Q, K, V, O, dO, LSE, dQ, dK, dV, nullptr, Ext{}, workspace, workspace_bytes, B, H, H_kv, S, D,
                  dtype, rope, rope_theta, rope_table, rope_table_rows, mask, window, alibi_slopes, softmax_scale,
                  stream);
}

int attnfuse_bwd_blocksparse(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                             const float* LSE, void* dQ, void* dK, void* dV,
                             const int* q_block_ptr, const int* k_block_idx,
                             const int* k_block_ptr, const int* q_block_idx,
                             void* workspace, size_t workspace_bytes,
                             int B, int H, int H_kv, int S, int D, int dtype,
                             int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                             int mask, int window,
                             const float* alibi_slopes, float softmax_scale, void* stream) {
  const int* m[] = {q_block_ptr, k_block_idx, k_block_ptr, q_block_idx};
  for (const int* x : m) if (!x || !aligned4(x)) return AF_ERR_INVALID_ARG;
  const void* outs[] = {dQ, dK, dV, workspace};
  for (const void* x : outs)
    for (const int* y : m) if (x == (const void*)y) return AF_ERR_INVALID_ARG;
  if (S < 1 || S > kMaxSparseS) return AF_ERR_INVALID_ARG;
  return bwd_impl(Q, K, V, O, dO, LSE, dQ, dK, dV, m, Ext{}, workspace, workspace_bytes, B, H, H_kv, S, D, dtype,
                  rope, rope_theta, rope_table, rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream);
}

int attnfuse_bwd_bias_norm(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                           const float* LSE, void* dQ, void* dK, void* dV,
                           const float* bias, long long bias_stride_b, long long bias_stride_h,
                           long long bias_stride_q, int norm,
                           void* workspace, size_t workspace_bytes,
                           int B, int H, int H_kv, int S, int D, int dtype,
                           int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                           int mask, int window,
                           const float* alibi_slopes, float softmax_scale, void* stream) {
  Ext e;
  e.bias = bias; e.sb = bias_stride_b; e.sh = bias_stride_h; e.sq = bias_stride_q; e.norm = norm;
  return bwd_impl(Q, K, V, O, dO, LSE, dQ, dK, dV, nullptr, e, workspace, workspace_bytes, B, H, H_kv, S, D, dtype,
                  rope, rope_theta, rope_table, rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream);
}

// ---------------------------------------------------------------- decode
size_t attnfuse_decode_workspace_bytes(int B, int H, int H_kv, int S_kv, int D) {
  if (B < 1 || H < 1 || H_kv < 1 || S_kv < 1 || S_kv > kMaxS || D < 2 || (D & 1) || H % H_kv) return 0;
  return decode_layout(B, H, H_kv, S_kv, D).total;
}

// The decode entry points share everything but where the partials live: the
// caller's workspace, or (workspace == nullptr) the library's static scratch.
static int decode_impl(const void* Q, const void* K, const void* V, const int* cache_lens, void* O, float* LSE,
                       void* workspace, size_t workspace_bytes, int B, int H, int H_kv, int S_kv, int D, int dtype,
                       int rope, float rope_theta, const float* rope_table, int rope_table_rows, int mask, int window,
                       const float* alibi_slopes, float softmax_scale, void* stream, bool static_scratch) {
  const void* ins[] = {Q, K, V};
  const void* outs[] = {O, LSE, workspace};
  const int nouts = static_scratch ? 2 : 3;
  for (const void* x : ins) if (!x || !aligned16(x)) return AF_ERR_INVALID_ARG;
  for (int i = 0; i < nouts; ++i) if (!outs[i] || !aligned16(outs[i])) return AF_ERR_INVALID_ARG;
  if (cache_lens && (reinterpret_cast<uintptr_t>(cache_lens) & 3u)) return AF_ERR_INVALID_ARG;
  for (int i = 0; i < nouts; ++i) {
    for (const void* y : ins) if (outs[i] == y) return AF_ERR_INVALID_ARG;
    if (outs[i] == static_cast<const void*>(cache_lens)) return AF_ERR_INVALID_ARG;
  }
  int rc = check_common(B, H, H_kv, S_kv, D, dtype, rope, rope_theta);
  if (rc != AF_OK) return rc;
  if ((rc = check_attn(mask, window, softmax_scale)) != AF_OK) return rc;
  if ((rc = check_table(rope, rope_table, rope_table_rows, S_kv, outs, nouts)) != AF_OK) return rc;
  const size_t need = attnfuse_decode_workspace_bytes(B, H, H_kv, S_kv, D);
  if (!static_scratch && workspace_bytes < need) return AF_ERR_INVALID_ARG;
  if (!supported_d(D) || dtype != AF_DTYPE_BF16 || H / H_kv > 32) return AF_ERR_UNSUPPORTED;
  if (static_scratch) {
    if (need > af::DECODE_SCRATCH_BYTES) return AF_ERR_TOO_LARGE;
    if (!(workspace = af::decode_scratch_ptr())) return AF_ERR_HIP;
  }

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
  p.table = (rope != AF_ROPE_NONE) ? reinterpret_cast<const float2*>(rope_table) : nullptr;
  return map_launch(af::launch_decode(D, rope, alibi_slopes != nullptr, p, st));
}

int attnfuse_decode(const void* Q, const void* K, const void* V, const int* cache_lens,
                    void* O, float* LSE, void* workspace, size_t workspace_bytes,
                    int B, int H, int H_kv, int S_kv, int D, int dtype,
                    int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                    int mask, int window,
                    const float* alibi_slopes, float softmax_scale, void* stream) {
  if (!workspace) return AF_ERR_INVALID_ARG;
  return decode_impl(Q, K, V, cache_lens, O, LSE, workspace, workspace_bytes, B, H, H_kv, S_kv, D, dtype, rope,
                     rope_theta, rope_table, rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream, false);
}

int attnfuse_decode_noalloc(const void* Q, const void* K, const void* V, const int* cache_lens,
                            void* O, float* LSE,
                            int B, int H, int H_kv, int S_kv, int D, int dtype,
                            int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                            int mask, int window,
                            const float* alibi_slopes, float softmax_scale, void* stream) {
  return decode_impl(Q, K, V, cache_lens, O, LSE, nullptr, 0, B, H, H_kv, S_kv, D, dtype, rope, rope_theta,
                     rope_table, rope_table_rows, mask, window, alibi_slopes, softmax_scale, stream, true);
}

static int rope_common(const void* X0, const void* X1, void* Y0, void* Y1, int B, int H, int H_kv, int S, int D,
                       int dtype, int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                       void* stream, bool inverse) {
  if (!X0 || !Y0 || !aligned16(X0) || !aligned16(Y0)) return AF_ERR_INVALID_ARG;
  if ((X1 == nullptr) != (Y1 == nullptr)) return AF_ERR_INVALID_ARG;
  if (X1 && (!aligned16(X1) || !aligned16(Y1))) return AF_ERR_INVALID_ARG;
  if (!X1) H_kv = 1;
  int rc = check_common(B, H, H_kv, S, D, dtype, rope, rope_theta);
  if (rc != AF_OK) return rc;
  if (rope == AF_ROPE_NONE) return AF_ERR_INVALID_ARG;
  const void* outs[] = {Y0, Y1};
  if ((rc = check_table(rope, rope_table, rope_table_rows, S, outs, 2)) != AF_OK) return rc;
  if (!supported_d(D)) return AF_ERR_UNSUPPORTED;
  hipStream_t st = static_cast<hipStream_t>(stream);
  af::RopeParams p{};
  p.x0 = X0; p.y0 = Y0; p.heads0 = H;
  p.x1 = X1; p.y1 = Y1; p.heads1 = X1 ? H_kv : 0;
  p.B = B; p.S = S;
  p.table = reinterpret_cast<const float2*>(rope_table);
  return map_launch(af::launch_rope(dtype == AF_DTYPE_FP32, D, rope, inverse, p, st));
}

int attnfuse_rope(const void* Q, const void* K, void* Qr, void* Kr, int B, int H, int H_kv, int S, int D,
                  int dtype, int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                  void* stream) {
  return rope_common(Q, K, Qr, Kr, B, H, H_kv, S, D, dtype, rope, rope_theta, rope_table, rope_table_rows, stream,
                     false);
}

int attnfuse_rope_bwd(const void* dQr, const void* dKr, void* dQ, void* dK, int B, int H, int H_kv, int S, int D,
                      int dtype, int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                      void* stream) {
  return rope_common(dQr, dKr, dQ, dK, B, H, H_kv, S, D, dtype, rope, rope_theta, rope_table, rope_table_rows, stream,
                     true);
}

}  // extern "C"
