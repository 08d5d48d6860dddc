/*
 * attnfuse.h -- C ABI of the MI355X (gfx950) fused RoPE + masked attention library.
 *
 * The method is AttnFuse (arXiv 2609.13612): attention whose query/key rotation
 * (RoPE, a pre-matmul transform) and score modifications (causal mask, sliding
 * window, ALiBi bias; post-matmul) run inside one online-softmax pass.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Layout.   Q, O, dO, dQ are [B, H, S, D]; K, V, dK, dV are [B, H_kv, S, D];
 *           LSE is [B, H, S]; all row-major and contiguous.  bf16 tensors hold
 *           IEEE bfloat16 bit patterns (2 bytes), fp32 tensors IEEE binary32.
 * Pointers. Every tensor pointer is a DEVICE pointer on the current HIP device,
 *           16-byte aligned.  ALiBi slopes are a device fp32 array [H].
 * Heads.    Query head h reads K/V head h / (H / H_kv) (grouped-query
 *           attention with contiguous groups); H must be a multiple of H_kv.
 * Positions 0..S-1 for queries and keys alike (self-attention, S_q = S_k = S).
 * Ownership The caller owns every buffer, including the RoPE cos/sin table
 *           (attnfuse_rope_table_fill) and the backward and decode workspaces.
 *           The library never allocates or frees device memory, keeps no state
 *           between calls and never synchronises: every entry point is a pure
 *           sequence of kernel launches, so any call may be captured in a HIP
 *           graph, including the first one.
 * RoPE      Every entry point that rotates takes rope_theta and a caller-owned
 * table     table of cos/sin values (below): rope_table, device fp32, filled
 *           by attnfuse_rope_table_fill with the same D and rope_theta, and
 *           rope_table_rows, the number of positions it was filled for, which
 *           must cover every position the call uses (S, or S_kv for decode).
 *           With AF_ROPE_NONE both are ignored and may be NULL / 0.
 * Streams.  All work is enqueued on `stream` (a hipStream_t; NULL = default
 *           stream) and runs asynchronously.
 * Errors.   Arguments are validated before any HIP call; no C++ exception
 *           crosses the ABI.  Return codes:
 *             AF_OK               success (work enqueued)
 *             AF_ERR_INVALID_ARG  bad pointer, size, enum or scalar
 *             AF_ERR_UNSUPPORTED  valid request with no compiled kernel
 *                                 (e.g. D not in {64, 128}, fp32 backward)
 *             AF_ERR_HIP          a HIP runtime call or kernel launch failed
 *             AF_ERR_TOO_LARGE    the request needs more than the static
 *                                 scratch of attnfuse_decode_noalloc
 *           attnfuse_strerror() maps a code to text.
 */
#ifndef ATTNFUSE_H
#define ATTNFUSE_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element type of Q, K, V, O, dO, dQ, dK, dV.  fp32 is the debug path: same
 * method, fp32 arithmetic throughout, no MFMA, one row per thread. */
enum { AF_DTYPE_BF16 = 0, AF_DTYPE_FP32 = 1 };

/* RoPE pairing (Section 4.1 "Fused RoPE": the paper's NeoX convention pairs
 * dimension i with i + D/2; interleaved pairs 2i with 2i+1).  Pair i rotates by
 * position * omega_i, omega_i = rope_theta^(-2i/D); the second element of a
 * pair gets +sin:  x_a' = x_a cos - x_b sin,  x_b' = x_a sin + x_b cos. */
enum { AF_ROPE_NONE = 0, AF_ROPE_NEOX = 1, AF_ROPE_INTERLEAVED = 2 };

/* Mask (Section 3.1 combinators full / causal / sliding_window).  Query i sees
 * key j when: NONE always; CAUSAL j <= i; SLIDING_WINDOW i - window < j <= i
 * (window keys, the diagonal included). */
enum { AF_MASK_NONE = 0, AF_MASK_CAUSAL = 1, AF_MASK_SLIDING_WINDOW = 2 };

/* Normalisation of the scores (Section 3.1 combinators softmax and
 * relu_attention): SOFTMAX as everywhere else; RELU uses P_ij = max(s_ij, 0)
 * with no normalisation and no row statistic (see attnfuse_fwd_bias_norm). */
enum { AF_NORM_SOFTMAX = 0, AF_NORM_RELU = 1 };

enum { AF_OK = 0, AF_ERR_INVALID_ARG = -1, AF_ERR_UNSUPPORTED = -2, AF_ERR_HIP = -3, AF_ERR_TOO_LARGE = -4 };

/*
 * RoPE cos/sin table (Section 4.1 "Fused RoPE": the rotation angle of pair i
 * at position n is n * omega_i with omega_i = rope_theta^(-2i/D), the RoFormer
 * frequencies).  The table holds rows x D/2 pairs of fp32 (cos, sin):
 *     T[n][i] = (cos(n * omega_i), sin(n * omega_i)),  n < rows, i < D/2,
 * each computed in fp64 and rounded once to fp32.  The caller allocates
 * attnfuse_rope_table_bytes(rows, D) bytes of device memory (16-byte
 * aligned), fills it once with attnfuse_rope_table_fill (one kernel launch on
 * `stream`; the table is valid for work ordered after it on the device), and
 * passes it, read only, to every RoPE call with the same D and rope_theta for
 * as long as it likes.  A table of R rows serves every call with S <= R.
 *
 * attnfuse_rope_table_bytes returns 0 for rows < 1, rows > 2^20 or an odd or
 * non-positive D.  attnfuse_rope_table_fill returns AF_ERR_INVALID_ARG for a
 * NULL or unaligned table, those sizes, or rope_theta not finite and > 0;
 * AF_ERR_UNSUPPORTED for D not in {64, 128}; AF_ERR_HIP if the launch fails.
 */
size_t attnfuse_rope_table_bytes(int rows, int D);
int attnfuse_rope_table_fill(float* table, int rows, int D, float rope_theta, void* stream);

/*
 * Fused forward (Section 2 online softmax; Section 4.1 fused RoPE; Section 3.1
 * score modifications; Section 4.4 saved row statistic).  Computes
 *     s_ij  = softmax_scale * <R_i q_i, R_j k_j> - slope_h * (i - j)
 *     O_i   = sum_j softmax_j(s_ij over visible j) v_j
 *     LSE_i = ln sum_{visible j} exp(s_ij)
 * where R_p is the RoPE rotation at position p (identity for AF_ROPE_NONE)
 * and the slope term is present only when alibi_slopes != NULL.
 *
 *   Q [B,H,S,D], K/V [B,H_kv,S,D]   inputs (dtype)
 *   O [B,H,S,D]                     output (dtype); must not alias an input
 *   LSE [B,H,S] fp32                output, natural log; a row with no visible
 *                                   key gets O = 0, LSE = -inf
 *   B, H, H_kv, S >= 1; H % H_kv == 0; D in {64, 128} (others: UNSUPPORTED)
 *   dtype       AF_DTYPE_*
 *   rope        AF_ROPE_*; rope_theta > 0 and finite when rope != NONE
 *   rope_table, rope_table_rows   the caller's cos/sin table for D and
 *               rope_theta with rope_table_rows >= S (used when rope != NONE)
 *   mask        AF_MASK_*; window >= 1 when SLIDING_WINDOW (ignored otherwise)
 *   alibi_slopes  device fp32 [H] or NULL
 *   softmax_scale finite, > 0 (typically 1/sqrt(D))
 *
 * Precision and range (bf16): without RoPE the bf16 inputs feed Q K^T
 * exactly; with RoPE the rotated Q' and K' are rounded to fp16 (11-bit
 * significand) for the score product, so |R q| and |R k| must stay below the
 * fp16 maximum 65504, and each score may move by up to
 * softmax_scale * sum_d |q'_d k'_d| * 2^-10: LSE_i then lies within the
 * largest such amount over row i's visible keys of the exact value (about
 * 1e-3 at softmax_scale = 1/sqrt(D) for unit-variance inputs, proportionally
 * more at larger scales or norms).  P and V meet in a bf16 product;
 * accumulation is fp32.
 */
int attnfuse_fwd(const void* Q, const void* K, const void* V, void* O, float* LSE,
                 int B, int H, int H_kv, int S, int D, int dtype,
                 int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                 int mask, int window,
                 const float* alibi_slopes, float softmax_scale, void* stream);

/* Bytes of device workspace attnfuse_bwd needs for these sizes and RoPE kind
 * (each part rounded up to a multiple of 256 bytes):
 *   8*B*H*S                  per query row: the softmax backward's row term
 *                            delta_i and LSE_i in log2 units (fp32 each)
 * + 2*B*H*S*D                sigma * dO converted once to fp16
 * + 4*B*H_kv                 sigma per (batch, K/V head): the power of two
 *                            that brings the group's largest |dO| into [1, 2)
 * + 4*B*H_kv*ceil(H/H_kv*S*D / 16384)   partial maxima of |dO|
 * + 2*(B*H + B*H_kv)*S*D     with RoPE only: Q' = R Q and K' = R K, rotated
 *                            once and rounded to fp16
 * Returns 0 for invalid sizes. */
size_t attnfuse_bwd_workspace_bytes(int B, int H, int H_kv, int S, int D, int rope);

/*
 * Backward of attnfuse_fwd (Section 4.4: no atomics -- a preprocessing pass,
 * a dQ pass over key tiles and a dK/dV pass over query tiles; probabilities
 * are re-derived from the saved LSE).  The preprocessing pass computes the
 * row statistics and, with RoPE, rotates Q and K once into the workspace (both
 * later passes read every tile many times, so rotating once is cheaper than
 * re-rotating per visit); the gradients leave through the inverse rotation:
 * dQ = R^T dQ', dK = R^T dK'.  For grouped-query attention dK and dV sum over
 * the H/H_kv query heads of their group.
 *
 * The softmax backward's row term delta_i = sum_j P_ij dP_ij: the dQ pass
 * uses rowsum(dO_i * O_i) of the O it is given (equal for the exact O) and
 * forms sum_j P_ij dP_ij itself, in fp32, for the dK/dV pass.
 *
 * Precision and range (bf16): the score, dV, dK and dQ products run on fp16
 * MFMA operands with fp32 accumulation.  dO enters them multiplied by sigma,
 * a power of two per (batch, K/V head) that brings the group's largest |dO|
 * into [1, 2), and the gradients leave divided by it, so the result is the
 * same at any scale of dO (exact power-of-two scaling).  The rotated |Q'| and
 * |K'| (as in attnfuse_fwd) and |V| must stay below the fp16 maximum 65504,
 * and max|V| below 16376 / D (128 at D = 128), which bounds the scaled
 * |dS| <= 4 D max|V| by the same maximum.
 *
 *   Q, K, V, O, dO, LSE  as produced/consumed by attnfuse_fwd with the same
 *                        variant arguments (LSE must be the forward's)
 *   dQ [B,H,S,D], dK/dV [B,H_kv,S,D]  outputs (dtype), fully overwritten; must
 *                        not alias inputs
 *   workspace            device memory of >= attnfuse_bwd_workspace_bytes(B,
 *                        H, H_kv, S, D, rope) bytes (16-byte aligned),
 *                        caller-owned scratch, overwritten
 *   other arguments      as attnfuse_fwd.  AF_DTYPE_FP32 runs the fp32 debug
 *                        backward (same passes, fp32 arithmetic; it uses only
 *                        the workspace's row statistics).
 */
int attnfuse_bwd(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                 const float* LSE, void* dQ, void* dK, void* dV,
                 void* workspace, size_t workspace_bytes,
                 int B, int H, int H_kv, int S, int D, int dtype,
                 int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                 int mask, int window,
                 const float* alibi_slopes, float softmax_scale, void* stream);

/*
 * Block-sparse attention (Section 4.3 "Block-Sparse Attention"): the variant
 * attnfuse_fwd computes with an extra block-level visibility test.  Positions
 * are grouped into blocks of AF_SPARSE_BLOCK = 64 (nb = ceil(S / 64) blocks per
 * side); query i sees key j only when block (i / 64, j / 64) is active AND the
 * elementwise mask allows it.  The kernels iterate only over active blocks:
 * each workgroup gathers the union of its query blocks' active key blocks and
 * skips the rest, so the work is proportional to the active fraction.  A row
 * whose visible set is empty gets O = 0, LSE = -inf (and zero gradients).
 *
 * The mask is one compressed-sparse-row list shared by every batch and head:
 *   q_block_ptr  device int32 [nb + 1]: row r's active key blocks are
 *                k_block_idx[q_block_ptr[r] .. q_block_ptr[r+1]-1];
 *                q_block_ptr[0] = 0, non-decreasing
 *   k_block_idx  device int32 [q_block_ptr[nb]]: key-block indices in [0, nb)
 *                (any order, duplicates allowed; rows strictly ascending, the
 *                canonical form, are read fastest; entries outside [0, nb)
 *                are ignored)
 * Both 4-byte aligned, caller-owned, read only.  The pointer array must be a
 * valid CSR offset list: it is read on the device, and offsets outside
 * k_block_idx are not detected (the Python binding builds and checks it).
 * S <= 64 * 2048 = 131072; dtype AF_DTYPE_BF16 (fp32: AF_ERR_UNSUPPORTED).
 * Other arguments and results as attnfuse_fwd.
 */
#define AF_SPARSE_BLOCK 64
int attnfuse_fwd_blocksparse(const void* Q, const void* K, const void* V, void* O, float* LSE,
                             const int* q_block_ptr, const int* k_block_idx,
                             int B, int H, int H_kv, int S, int D, int dtype,
                             int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                             int mask, int window,
                             const float* alibi_slopes, float softmax_scale, void* stream);

/*
 * Backward of attnfuse_fwd_blocksparse (Section 4.3: the backward also visits
 * only active blocks).  The dQ pass walks each query block's key blocks (the
 * forward's list); the dK/dV pass walks each key block's query blocks, so it
 * also needs the transposed list of the same mask:
 *   k_block_ptr  device int32 [nb + 1], q_block_idx: key-block column c's
 *                active query blocks (compressed sparse column form)
 * The two lists must describe the same block set; no check is made that they
 * do.  Workspace, other arguments and results as attnfuse_bwd; bf16 only.
 */
int attnfuse_bwd_blocksparse(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                             const float* LSE, void* dQ, void* dK, void* dV,
                             const int* q_block_ptr, const int* k_block_idx,
                             const int* k_block_ptr, const int* q_block_idx,
                             void* workspace, size_t workspace_bytes,
                             int B, int H, int H_kv, int S, int D, int dtype,
                             int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                             int mask, int window,
                             const float* alibi_slopes, float softmax_scale, void* stream);

/*
 * attnfuse_fwd with the two remaining combinators of Section 3.1: a dense
 * additive bias tensor (additive_bias) and relu attention (relu_attention).
 * The paper names both without defining them; here
 *     s_ij  = softmax_scale * <R_i q_i, R_j k_j> + bias[b, h, i, j]
 * (added before the mask, like ALiBi), then with norm = AF_NORM_SOFTMAX the
 * usual O = softmax(s) V and LSE, and with norm = AF_NORM_RELU
 *     O_i = sum_{visible j} max(s_ij, 0) v_j
 * (no normalisation: a 1/n factor folds into softmax_scale and the bias), with
 * no row statistic: LSE is not written and may be NULL.
 *
 *   bias     device fp32, or NULL for none.  Element (b, h, i, j) -- batch,
 *            query head, query position, key position -- is read at
 *            bias[b*bias_stride_b + h*bias_stride_h + i*bias_stride_q + j]:
 *            keys contiguous, the other strides in elements, >= 0 (0
 *            broadcasts: e.g. a key-padding bias [B, 1, 1, S] has strides
 *            (S, 0, 0)).  4-byte aligned, read only, must not alias an
 *            output; the caller guarantees every addressed element exists.
 *   norm     AF_NORM_*
 *   other arguments as attnfuse_fwd.  Supported: bf16, D in {64, 128}, every
 *   RoPE kind and mask, without ALiBi (a bias tensor can carry it); other
 *   combinations return AF_ERR_UNSUPPORTED.  bias = NULL with
 *   AF_NORM_SOFTMAX is exactly attnfuse_fwd.
 */
int attnfuse_fwd_bias_norm(const void* Q, const void* K, const void* V, void* O, float* LSE,
                           const float* bias, long long bias_stride_b, long long bias_stride_h,
                           long long bias_stride_q, int norm,
                           int B, int H, int H_kv, int S, int D, int dtype,
                           int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                           int mask, int window,
                           const float* alibi_slopes, float softmax_scale, void* stream);

/*
 * Backward of attnfuse_fwd_bias_norm (the same bias and norm).  The bias gets
 * no gradient.  Under AF_NORM_RELU the probabilities are recomputed as
 * max(s, 0) and dS = dP where s > 0 (0 at s = 0); LSE is not used and may be
 * NULL.  Workspace, other arguments and results as attnfuse_bwd.
 */
int attnfuse_bwd_bias_norm(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                           const float* LSE, void* dQ, void* dK, void* dV,
                           const float* bias, long long bias_stride_b, long long bias_stride_h,
                           long long bias_stride_q, int norm,
                           void* workspace, size_t workspace_bytes,
                           int B, int H, int H_kv, int S, int D, int dtype,
                           int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                           int mask, int window,
                           const float* alibi_slopes, float softmax_scale, void* stream);

/*
 * Standalone rotation, the separate-RoPE path (Section 5.3 "The Rotation
 * Calculus": pre-rotation reads Q and K and writes Q' and K' once, an HBM round
 * trip, before an attention that has no RoPE).  One bandwidth-bound launch
 * rotates both tensors:  Qr = R Q,  Kr = R K  (positions 0..S-1).
 *
 *   Q [B,H,S,D] -> Qr;  K [B,H_kv,S,D] -> Kr  (dtype).  In-place is allowed
 *   (Qr == Q, Kr == K).  K and Kr may both be NULL to rotate Q alone (H_kv is
 *   then ignored).  rope must be NEOX or INTERLEAVED.  D in {64, 128}.
 *   rope_table / rope_table_rows as attnfuse_fwd (rows >= S); the table must
 *   not be an output.
 */
int attnfuse_rope(const void* Q, const void* K, void* Qr, void* Kr,
                  int B, int H, int H_kv, int S, int D, int dtype,
                  int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                  void* stream);

/* Inverse rotation (the separate path's backward): dQ = R^T dQr, dK = R^T dKr.
 * Same arguments and rules as attnfuse_rope. */
int attnfuse_rope_bwd(const void* dQr, const void* dKr, void* dQ, void* dK,
                      int B, int H, int H_kv, int S, int D, int dtype,
                      int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                      void* stream);

/* Bytes of device workspace attnfuse_decode needs: four partial (max, sum,
 * accumulator) triples per (sequence, query head, cache chunk), one per
 * first-phase wave, fp32.  The chunk length is a power of two in [128, 4096]
 * chosen from B * H_kv * S_kv so the first phase launches about 512
 * workgroups.  Returns 0 for invalid sizes. */
size_t attnfuse_decode_workspace_bytes(int B, int H, int H_kv, int S_kv, int D);

/*
 * Decode attention over a key/value cache (Section 4.2 "Flash Decoding"): one
 * query per sequence.  Phase 1 splits each sequence's cache into chunks,
 * each streamed by four waves, and computes a partial online-softmax triple
 * (m, l, acc) per wave for all query heads of a K/V head at once (the group's
 * heads fill the MFMA's columns by cyclic replication, so K and V are read
 * exactly once); phase 2 merges the partials by log-sum-exp.  With L = cache_lens[b] the query sits at position
 * p = L - 1 and
 *     s_j = softmax_scale * <R_p q, k_j> - slope_h * (p - j),   j < L
 *     O   = softmax_j(s_j over visible j) v_j,   LSE = ln sum_{visible j} exp(s_j)
 * The cache holds keys ALREADY ROTATED at their own positions (rotate them once
 * when they are written, e.g. with attnfuse_rope); only the query is rotated
 * here.  Under RoPE the rotated query and the cached keys meet in fp16, as in
 * attnfuse_fwd, so |k| must stay below the fp16 maximum.
 *
 *   Q [B,H,D]                    the newest token's queries (dtype), unrotated
 *   K, V [B,H_kv,S_kv,D]         the caches (dtype), row-major, contiguous
 *   cache_lens                   device int32 [B] or NULL (every sequence uses
 *                                S_kv entries); values above S_kv are clamped
 *                                to S_kv, values below 1 give O = 0, LSE = -inf
 *   O [B,H,D] (dtype), LSE [B,H] fp32 (natural log)
 *   workspace                    device memory of >= attnfuse_decode_workspace_
 *                                bytes(B, H, H_kv, S_kv, D) bytes, caller-owned
 *   mask                         NONE or CAUSAL: every cached key is visible
 *                                (all precede the query); SLIDING_WINDOW: the
 *                                last `window` keys
 *   rope, rope_theta, rope_table, alibi_slopes, softmax_scale   as
 *                                attnfuse_fwd (rope_table_rows >= S_kv)
 *   dtype                        AF_DTYPE_BF16 only; D in {64, 128};
 *                                H / H_kv <= 32 (else AF_ERR_UNSUPPORTED)
 */
int attnfuse_decode(const void* Q, const void* K, const void* V, const int* cache_lens,
                    void* O, float* LSE, void* workspace, size_t workspace_bytes,
                    int B, int H, int H_kv, int S_kv, int D, int dtype,
                    int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                    int mask, int window,
                    const float* alibi_slopes, float softmax_scale, void* stream);

/*
 * attnfuse_decode for callers that cannot allocate device memory: code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation.
 * Same computation and arguments, without the workspace: the partials live in
 * a static device buffer of AF_DECODE_SCRATCH_BYTES (32 MiB) that the library
 * holds on every GPU it runs on until the process ends (its address is looked
 * up once per device, on the first call there).  Requests for which
 * attnfuse_decode_workspace_bytes exceeds it return AF_ERR_TOO_LARGE (use
 * attnfuse_decode with a workspace).  Nothing needs clearing between calls
 * (every partial is written before it is read), but every call on one GPU uses
 * that GPU's one buffer: calls that may overlap on a GPU (on different streams
 * or from several threads) race and must be ordered by the caller.
 */
#define AF_DECODE_SCRATCH_BYTES (32u << 20)
int attnfuse_decode_noalloc(const void* Q, const void* K, const void* V, const int* cache_lens,
                            void* O, float* LSE,
                            int B, int H, int H_kv, int S_kv, int D, int dtype,
                            int rope, float rope_theta, const float* rope_table, int rope_table_rows,
                            int mask, int window,
                            const float* alibi_slopes, float softmax_scale, void* stream);

/* Static text for a return code (never NULL). */
const char* attnfuse_strerror(int code);

/* ABI version; bumped on any incompatible change. */
int attnfuse_version(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTNFUSE_H */
