// Decode attention over a key/value cache, bf16 inputs, MFMA with fp32
// accumulation, for gfx950 (Section 4.2 "Flash Decoding"; Table tab:decode).
//
// One query per sequence makes the work a stream over the cache: each K/V
// element is used once per query head of its group, so the kernel is bound by
// HBM and is built to read the cache exactly once at full width.
//
// Phase 1 (decode_split_kernel): workgroup = 4 waves = one (sequence, K/V
//   head, chunk of `chunk` keys); the four waves take the chunk's 32-key
//   tiles in turn, so the workgroup streams its chunk front to back.  Scores
//   are formed transposed, S^T = K Q'^T: the 32 MFMA columns are the group's
//   query heads, replicated cyclically when the group has fewer than 32 (K and
//   V are then read once for all of them); every lane owns one head column, so
//   the softmax statistics stay in-lane as in the prefill kernel.  K tiles go
//   from HBM straight into registers as the A operand (lane = key row); V
//   tiles go through the wave's own LDS tile for the transpose read of
//   O^T += V^T P^T.  The first tile's loads are issued before the query is
//   loaded and rotated; each next tile's as soon as the current tile's score
//   MFMAs have consumed its keys, so one tile per wave is always in flight.
//   The register budget is held to two waves per SIMD so that two workgroups
//   stream on every CU at once.  Each wave then writes its own (m, l, acc)
//   partial for the group's G query heads straight from its registers (the
//   kernel has no barrier); chunks with no visible key return at once.
// Phase 2 (decode_combine_kernel): per (sequence, head), merge the wave
//   partials of the chunks that hold visible keys by log-sum-exp and write O
//   and LSE; the head's dims are spread over several workgroups so the merge
//   reads the partials with the whole chip, in one round trip to memory.
//
// Precision: without RoPE the bf16 query and keys meet exactly in a bf16
// MFMA.  With RoPE the query is rotated at position L-1 in fp32 and rounded to
// fp16, and the (already rotated) bf16 cache keys are widened to fp16 in
// registers (exact inside the fp16 range), as the prefill kernel does for its
// rotated operands.  P and V are bf16.
#include <atomic>

#include "common.hpp"
#include "launch.hpp"

// Device memory for the partials of callers that cannot allocate
// (attnfuse_decode_noalloc): one file-scope array, which every device the
// library runs on holds until the process ends.  In host code its name stands
// for a host-side shadow, not a device address; decode_scratch_ptr() looks the
// address up once per device and keeps it, and only that address is used.
static __device__ __align__(256) unsigned char scratch[af::DECODE_SCRATCH_BYTES];

namespace af {

namespace {
constexpr int kMaxScratchDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxScratchDevices];   // per device, resolved on first use
}  // namespace

void* decode_scratch_ptr() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return nullptr;
  void* ptr = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (ptr) return ptr;
  if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
  g_scratch_ptr[dev].store(ptr, std::memory_order_release);
  return ptr;
}

template <int D>
struct DecCfg {
  static constexpr int NW = 4;                      // waves per workgroup
  static constexpr int KS = D / 16;                 // MFMA k-steps over the head dimension
  static constexpr int MT = D / 32;                 // 32-row output tiles over the head dimension
  static constexpr int VP = D + 16;                 // V tile pitch (transpose reads)
  static constexpr int VT = 32 * VP;                // one wave's V tile (elements)
  static constexpr int VPL = 32 * (D / 8) / 64;     // 16-byte V chunks per lane per tile
  static constexpr int SMEM = NW * VT;              // uint16 elements
};

__device__ __forceinline__ int seq_len(const DecodeParams& p, int b) {
  return p.lens ? min(p.lens[b], p.S) : p.S;
}

// First visible key of a sequence with L cached keys.
__device__ __forceinline__ int first_key(const DecodeParams& p, int L) {
  return (p.window > 0) ? max(0, L - p.window) : 0;
}

template <int D, int ROPE, bool ALIBI>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2)))
void decode_split_kernel(DecodeParams p) {
  using C = DecCfg<D>;
  constexpr bool QF16 = ROPE != ROPE_NONE;
  __shared__ __attribute__((aligned(16))) uint16_t smem[C::SMEM];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lq = lane & 31, lg = lane >> 5;
  const int split = (int)(blockIdx.x % p.nsplit);
  const int unit = (int)(blockIdx.x / p.nsplit);
  const int b = unit / p.Hkv, g = unit % p.Hkv;
  const int G = p.H / p.Hkv;
  const int L = seq_len(p, b);
  if (L < 1) return;
  const int lo = first_key(p, L);
  const int c0 = split * p.chunk;
  if (c0 + p.chunk <= lo || c0 >= L) return;       // no visible key in this chunk (workgroup-uniform)
  const int pos = L - 1;                           // the query's position

  const int hc = lq % G;                           // head of this lane's column (cyclic replication)
  const int h = g * G + hc;
  const uint16_t* __restrict__ K = static_cast<const uint16_t*>(p.k) + (size_t)unit * p.S * D;
  const uint16_t* __restrict__ V = static_cast<const uint16_t*>(p.v) + (size_t)unit * p.S * D;

  const float c2 = p.scale * kLog2e;
  const float slope2 = ALIBI ? p.slopes[h] * kLog2e : 0.f;

  // This wave's tiles: every NW-th tile of the chunk from the wave's own,
  // starting at the first tile that holds a visible key.
  constexpr int STEP = 32 * C::NW;
  const int first = lo & ~31;
  const int kend = min(c0 + p.chunk, L);
  int kbeg = c0 + 32 * wave;
  if (kbeg < first) kbeg += (first - kbeg + STEP - 1) / STEP * STEP;

  uint16_t* Vw = smem + wave * C::VT;
  const int tr_key = 4 * lg + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);

  f32x16 acc[C::MT];
#pragma unroll
  for (int i = 0; i < C::MT; ++i) acc[i] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  u32x4 kreg[C::KS], vreg[C::VPL];
  auto load_tile = [&](int n0) {   // rows past L are clamped to L-1 (finite data, masked)
    const int n = min(n0 + lq, L - 1);
#pragma unroll
    for (int s = 0; s < C::KS; ++s) kreg[s] = ld16(K + (size_t)n * D + 16 * s + 8 * lg);
#pragma unroll
    for (int i = 0; i < C::VPL; ++i) {
      const int it = lane + 64 * i;
      const int r = it / (D / 8), c = it % (D / 8);
      vreg[i] = ld16(V + (size_t)min(n0 + r, L - 1) * D + 8 * c);
    }
  };

  if (kbeg < kend) load_tile(kbeg);
  // Query operand (B of S^T = K Q'^T): lane holds head column hc, dims 16s + 8lg .. +7.
  const uint16_t* __restrict__ Qh = static_cast<const uint16_t*>(p.q) + ((size_t)b * p.H + h) * D;
  u32x4 qreg[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) qreg[s] = ld16(Qh + 16 * s + 8 * lg);
  if constexpr (ROPE == ROPE_NEOX) {
#pragma unroll
    for (int s = 0; s < C::KS / 2; ++s)
      rotate_neox8<false, true>(qreg[s], qreg[s + C::KS / 2], p.table + (size_t)pos * (D / 2) + 16 * s + 8 * lg);
  } else if constexpr (ROPE == ROPE_INTERLEAVED) {
#pragma unroll
    for (int s = 0; s < C::KS; ++s)
      rotate_interleaved8<false, true>(qreg[s], p.table + (size_t)pos * (D / 2) + 8 * s + 4 * lg);
  }

  for (int n0 = kbeg; n0 < kend; n0 += STEP) {
    // V tile to this wave's LDS tile (the previous tile's transpose reads,
    // issued earlier by this wave, complete first: LDS is in order per wave)
#pragma unroll
    for (int i = 0; i < C::VPL; ++i) {
      const int it = lane + 64 * i;
      const int r = it / (D / 8), c = it % (D / 8);
      *reinterpret_cast<u32x4*>(Vw + r * C::VP + 8 * c) = vreg[i];
    }
    if constexpr (QF16) {   // cached keys bf16 -> fp16 to meet the fp16 query
#pragma unroll
      for (int s = 0; s < C::KS; ++s)
#pragma unroll
        for (int w = 0; w < 4; ++w) kreg[s][w] = pack_f16(bf_lo(kreg[s][w]), bf_hi(kreg[s][w]));
    }
    f32x16 st = f32x16{};
#pragma unroll
    for (int s = 0; s < C::KS; ++s) st = mfma32<QF16>(kreg[s], qreg[s], st);
    if (n0 + STEP < kend) load_tile(n0 + STEP);

    // element r: key n0 + 8 (r/4) + 4 lg + r%4 of head column lq
    if constexpr (ALIBI) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + 8 * (r >> 2) + 4 * lg + (r & 3);
        st[r] = __builtin_fmaf(st[r], c2, slope2 * (float)(n - pos));
      }
    }
    if (n0 + 32 > L || n0 < lo) {   // wave-uniform: edge tiles only
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int n = n0 + 8 * (r >> 2) + 4 * lg + (r & 3);
        st[r] = (n < L && n >= lo) ? st[r] : -INFINITY;
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, st[r]);
    mx = pair_max(mx);
    if constexpr (!ALIBI) mx *= c2;
    const float m_new = fmaxf(m_run, mx);
    if (__any(m_new > m_run + 8.f)) {   // raise the reference max (wave-uniform)
      const float alpha = (m_run == -INFINITY) ? 0.f : fast_exp2(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < C::MT; ++i) acc[i] *= alpha;
      m_run = m_new;
    }
    const float m_use = (m_run == -INFINITY) ? 0.f : m_run;
    float pv[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      pv[r] = fast_exp2(ALIBI ? (st[r] - m_use) : __builtin_fmaf(st[r], c2, -m_use));
      l_run += pv[r];
    }
    u32x4 pop[2];
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int w = 0; w < 4; ++w) pop[hf][w] = pack_bf16(pv[8 * hf + 2 * w], pv[8 * hf + 2 * w + 1]);

    // O^T += V^T P^T (V^T from transpose reads of the row-major V tile)
#pragma unroll
    for (int hf = 0; hf < 2; ++hf)
#pragma unroll
      for (int mt = 0; mt < C::MT; ++mt) {
        const uint16_t* base = Vw + (16 * hf + tr_key) * C::VP + 32 * mt + tr_col;
        const u32x2 lo2 = lds_read_tr16(base);
        const u32x2 hi2 = lds_read_tr16(base + 8 * C::VP);
        const u32x4 a = {lo2[0], lo2[1], hi2[0], hi2[1]};
        acc[mt] = mfma32(a, pop[hf], acc[mt]);
      }
  }

  // One partial per wave, straight from registers: the first G head columns.
  const float l_tot = pair_sum(l_run);
  const int nslot = p.nsplit * C::NW;
  if (lq < G) {
    const size_t prow = ((size_t)b * p.H + g * G + lq) * nslot + split * C::NW + wave;
    float* dst = p.part_acc + prow * D + 4 * lg;
#pragma unroll
    for (int mt = 0; mt < C::MT; ++mt)
#pragma unroll
      for (int a = 0; a < 4; ++a)
        *reinterpret_cast<float4*>(dst + 32 * mt + 8 * a) =
            float4{acc[mt][4 * a], acc[mt][4 * a + 1], acc[mt][4 * a + 2], acc[mt][4 * a + 3]};
    if (lg == 0) {
      p.part_ml[prow * 2] = m_run;
      p.part_ml[prow * 2 + 1] = l_tot;
    }
  }
}

// Fold the (max, sum) pair (m2, l2) into the running pair (m, l), log2 units.
__device__ __forceinline__ void merge_ml(float& m, float& l, float m2, float l2) {
  const float M = fmaxf(m, m2);
  if (M == -INFINITY) return;
  l = l * fast_exp2(m - M) + l2 * fast_exp2(m2 - M);
  m = M;
}

// Phase 2.  Workgroup = 256 threads = one (sequence, query head) and 32 of its
// dims, as eight groups of 32 threads that each take every eighth partial (4
// per chunk, one per wave).  Each thread loads its first PF partials'
// accumulators and maxima together with the statistics, so the merge costs
// one round trip to memory: each thread folds the (m, l) pairs it reads into
// a running pair, the pairs merge across the workgroup, and every thread
// weights its accumulators by 2^(m_s - M).
template <int D, int PF>
__global__ __launch_bounds__(256) void decode_combine_kernel(DecodeParams p) {
  __shared__ float red[256];
  __shared__ float wred[8];
  const int bh = blockIdx.x, t = threadIdx.x, lane = t & 63, wv = t >> 6;
  const int d = 32 * blockIdx.y + (t & 31), grp = t >> 5;
  const int b = bh / p.H;
  const int L = seq_len(p, b);
  uint16_t* O = static_cast<uint16_t*>(p.o) + (size_t)bh * D;
  if (L < 1) {   // workgroup-uniform
    if (grp == 0) O[d] = 0;
    if (t == 0 && blockIdx.y == 0) p.lse[bh] = -INFINITY;
    return;
  }
  constexpr int NWV = DecCfg<D>::NW;   // partials per chunk
  const int nslot = p.nsplit * NWV;
  const int s_lo = first_key(p, L) / p.chunk, s_hi = (L - 1) / p.chunk;
  const int n = (s_hi - s_lo + 1) * NWV;
  const float* ml = p.part_ml + ((size_t)bh * nslot + s_lo * NWV) * 2;
  const float* acc = p.part_acc + ((size_t)bh * nslot + s_lo * NWV) * D + d;
  float a[PF], mm[PF];
#pragma unroll
  for (int j = 0; j < PF; ++j) {
    const int i = grp + 8 * j;
    a[j] = (i < n) ? acc[(size_t)i * D] : 0.f;
    mm[j] = (i < n) ? ml[2 * i] : -INFINITY;
  }
  float m = -INFINITY, l = 0.f;
  for (int i = t; i < n; i += 256) {
    const float2 v = *reinterpret_cast<const float2*>(ml + 2 * i);
    merge_ml(m, l, v.x, v.y);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) merge_ml(m, l, __shfl_xor(m, o), __shfl_xor(l, o));
  if (lane == 0) {
    wred[2 * wv] = m;
    wred[2 * wv + 1] = l;
  }
  __syncthreads();
  m = wred[0];
  l = wred[1];
#pragma unroll
  for (int w = 1; w < 4; ++w) merge_ml(m, l, wred[2 * w], wred[2 * w + 1]);
  float o = 0.f;
#pragma unroll
  for (int j = 0; j < PF; ++j) o += a[j] * fast_exp2(mm[j] - m);
  for (int i = grp + 8 * PF; i < n; i += 8) o += acc[(size_t)i * D] * fast_exp2(ml[2 * i] - m);
  red[t] = o;
  __syncthreads();
  if (grp == 0) {
    float sum = 0.f;
#pragma unroll
    for (int g = 0; g < 8; ++g) sum += red[32 * g + t];
    O[d] = static_cast<uint16_t>(pack_bf16(sum / l, 0.f) & 0xffffu);
    if (t == 0 && blockIdx.y == 0) p.lse[bh] = (m + __log2f(l)) * kLn2;
  }
}

template <int D, int ROPE, bool ALIBI>
static int launch_one(const DecodeParams& p, hipStream_t st) {
  const long long blocks = (long long)p.nsplit * p.B * p.Hkv;
  hipLaunchKernelGGL((decode_split_kernel<D, ROPE, ALIBI>), dim3((unsigned)blocks), dim3(256), 0, st, p);
  // preload depth: every partial of a head (8 groups x PF) when it fits
  const dim3 cgrid((unsigned)(p.B * p.H), D / 32);
  if (p.nsplit * DecCfg<D>::NW <= 8 * 16)
    hipLaunchKernelGGL((decode_combine_kernel<D, 16>), cgrid, dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL((decode_combine_kernel<D, 32>), cgrid, dim3(256), 0, st, p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// The mask is a runtime lower bound on the key index (p.window > 0 for a
// sliding window): NONE and CAUSAL see the same keys in decode.
template <int D>
static int dispatch_rope(int rope, bool alibi, const DecodeParams& p, hipStream_t st) {
  switch (rope) {
    case ROPE_NONE: return alibi ? launch_one<D, ROPE_NONE, true>(p, st) : launch_one<D, ROPE_NONE, false>(p, st);
    case ROPE_NEOX: return alibi ? launch_one<D, ROPE_NEOX, true>(p, st) : launch_one<D, ROPE_NEOX, false>(p, st);
    case ROPE_INTERLEAVED:
      return alibi ? launch_one<D, ROPE_INTERLEAVED, true>(p, st) : launch_one<D, ROPE_INTERLEAVED, false>(p, st);
  }
  return -2;
}

int launch_decode(int D, int rope, bool alibi, const DecodeParams& p, hipStream_t st) {
  if (D == 64) return dispatch_rope<64>(rope, alibi, p, st);
  if (D == 128) return dispatch_rope<128>(rope, alibi, p, st);
  return -2;
}

}  // namespace af
