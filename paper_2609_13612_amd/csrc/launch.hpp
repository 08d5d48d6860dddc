// Internal host-side interface between the C-ABI layer (api.cpp) and the
// kernel translation units.  Each launcher maps runtime enums onto one
// compile-time template instantiation and enqueues it on the given stream.
#pragma once
#include <hip/hip_runtime.h>

namespace af {

// Score-modification / normalisation variants beyond masks and ALiBi (the
// additive_bias and relu_attention combinators): a dense fp32 bias tensor
// added to the scaled scores, and P = max(s, 0) in place of the softmax.
enum { EXT_NONE = 0, EXT_BIAS = 1, EXT_RELU = 2, EXT_RELU_BIAS = 3 };

struct FwdParams {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  int B, H, Hkv, S, window;
  const float* slopes;    // [H] or nullptr
  float scale;
  const float2* table;    // [rows >= S][D/2] (cos, sin); nullptr without RoPE
  int heads_per_wg;       // set by the bf16 launcher: query heads packed per workgroup
  const int* bq_ptr;      // block-sparse mask by 64-row query block (CSR row pointers), or nullptr
  const int* bk_idx;      // and the active 64-key blocks of each row
  const float* bias;      // dense bias: element (b, h, i, j) at bias[b*bias_sb + h*bias_sh + i*bias_sq + j]
  long long bias_sb, bias_sh, bias_sq;
};

struct BwdParams {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dout;
  const float* lse;
  void* dq;
  void* dk;
  void* dv;
  float* delta;           // workspace [B*H*S]: sigma * delta_i (see dscale); rowsum(dO * O) from the
                          // preprocessing pass, replaced by sum_j P_ij dP_ij in the dQ pass
  float* lse2;            // workspace [B*H*S]: LSE in log2 units (+inf for empty rows)
  void* do16;             // workspace [B,H,S,D] fp16: sigma * dO
  float* dscale;          // workspace [B*H_kv]: sigma, a power of two per (batch, K/V head)
  uint32_t* dmax;         // workspace [B*H_kv*dmax_chunks]: partial max |dO| (bf16 magnitude bits)
  int dmax_chunks;        // partial maxima per (batch, K/V head)
  void* qr16;             // workspace [B,H,S,D] fp16: Q' = R Q (RoPE only, else nullptr)
  void* kr16;             // workspace [B,H_kv,S,D] fp16: K' = R K (RoPE only, else nullptr)
  int B, H, Hkv, S, window;
  const float* slopes;
  float scale;
  const float2* table;
  int heads_per_wg;       // set by the launcher for the dQ kernel
  const int* bq_ptr;      // block-sparse mask by 64-row query block (CSR), or nullptr
  const int* bk_idx;
  const int* bk_ptr;      // the same mask by 64-key block (CSC), or nullptr
  const int* bq_idx;
  const float* bias;      // dense bias, as in FwdParams
  long long bias_sb, bias_sh, bias_sq;
};

struct DecodeParams {
  const void* q;          // [B, H, D]
  const void* k;          // cache [B, H_kv, S, D], keys already rotated
  const void* v;          // cache [B, H_kv, S, D]
  const int* lens;        // device [B] cache lengths, or nullptr (all S)
  void* o;                // [B, H, D]
  float* lse;             // [B, H]
  float* part_ml;         // workspace [B, H, 4 nsplit, 2]: wave partial max and sum (log2 units)
  float* part_acc;        // workspace [B, H, 4 nsplit, D]: wave partial accumulator
  int B, H, Hkv, S;
  int window;             // > 0: sliding window of that many keys; 0: every cached key
  int chunk, nsplit;      // keys per phase-1 workgroup; chunks per sequence
  const float* slopes;
  float scale;
  const float2* table;
};

struct RopeParams {
  const void* x0;  void* y0;  int heads0;   // first tensor [B, heads0, S, D]
  const void* x1;  void* y1;  int heads1;   // optional second tensor (heads1 may be 0)
  int B, S;
  const float2* table;
};

// Return 0 on success, -2 when the variant is not compiled, -3 on a HIP error.
// ext: EXT_* (common.hpp); variants other than EXT_NONE run without ALiBi and block masks.
int launch_fwd_bf16(int D, int rope, int mask, bool alibi, int ext, const FwdParams& p, hipStream_t st);
int launch_fwd_fp32(int D, int rope, int mask, bool alibi, const FwdParams& p, hipStream_t st);
int launch_bwd_bf16(int D, int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st);
// The dK/dV pass alone (the last launch of launch_bwd_bf16).
int launch_bwd_dkdv_bf16(int D, int rope, int mask, bool alibi, int ext, const BwdParams& p, hipStream_t st);
int launch_bwd_fp32(int D, int rope, int mask, bool alibi, const BwdParams& p, hipStream_t st);
int launch_decode(int D, int rope, bool alibi, const DecodeParams& p, hipStream_t st);
int launch_rope(bool fp32, int D, int rope, bool inverse, const RopeParams& p, hipStream_t st);
int launch_rope_table(float2* table, int rows, int D, double theta, hipStream_t st);

// Static device scratch of the decode entry point that allocates nothing: its
// size, and its address on the current device (nullptr if it cannot be found).
constexpr size_t DECODE_SCRATCH_BYTES = (size_t)32 << 20;
void* decode_scratch_ptr();

}  // namespace af
