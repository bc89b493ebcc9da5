// Important-token selection (Sec. 2 item 1): tokens are chosen by the
// deviation of their freshly computed keys from the offline cached keys,
// aggregated over several early layers (typically the 2nd to the 4th). Score of
// a document token = mean over the selection layers of the L2 norm of
// (k_fresh - k_cached) over all its KV heads and features; request b keeps its
// n_b highest-scoring tokens (equal scores: lower index first), listed in
// ascending original order, which is the idx every other entry point takes.
//
// select_score_kernel: one wave per document row, HBM-bound (2 * layers * row
// bytes read per row); every lane loads 16-byte pieces of the row for all
// layers before reducing, fp32 sums of squares, a wave reduction per layer.
//
// select_topn_kernel: one 1024-thread workgroup per request, the keys held in
// registers (32 per lane, slab by slab beyond 32k tokens). Scores are
// non-negative floats, so their bit patterns order like the values: a radix
// select over 8-bit digits finds the key T of the n-th highest score and how
// many tokens scoring exactly T to keep. The digit histogram is kept in 32
// copies, one per lane of a half wave (rows padded to 257 words so that one
// digit's copies sit in different banks): scores cluster, and with a single
// copy the lanes of one instruction that share a digit serialise on its word. The passes start below the bits that
// the lowest and highest key share, so the first histogram spreads over the
// scores' actual range, and stop early once a digit's keys are all taken.
// Each wave owns a contiguous range of tokens; a prefix sum over the waves of
// their kept counts, then ballots within each wave, place every kept index, so
// the output comes out sorted.
#include "daf_internal.h"

namespace daf {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kScoreThreads = 256;
constexpr int kTopnThreads = 1024;
constexpr int kTopnWaves = kTopnThreads / 64;
constexpr int kHistCopies = 32, kHistStride = 257;

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

// Sum of squared differences of the 16-byte pieces a and b (8 bf16 or 4 fp32).
template <bool BF16>
__device__ __forceinline__ float sq_diff(u32x4 a, u32x4 b) {
  float s = 0.f;
  if (BF16) {
    const bf16x8 x = __builtin_bit_cast(bf16x8, a), y = __builtin_bit_cast(bf16x8, b);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float d = (float)x[i] - (float)y[i];
      s = __builtin_fmaf(d, d, s);
    }
  } else {
    // whole-vector casts: a bit cast of a vector element expression reads the
    // vector's first element
    const f32x4 x = __builtin_bit_cast(f32x4, a), y = __builtin_bit_cast(f32x4, b);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float d = x[i] - y[i];
      s = __builtin_fmaf(d, d, s);
    }
  }
  return s;
}

// CPL = 16-byte pieces per lane (row bytes / 1024, rounded up).
template <bool BF16, int CPL>
__global__ __launch_bounds__(kScoreThreads) void select_score_kernel(const SelectLaunch p) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * (kScoreThreads / 64) + (threadIdx.x >> 6);
  if (row >= p.rows) return;
  const int pieces = p.row_bytes / 16;
  float acc = 0.f;
  for (int l0 = 0; l0 < p.n_layers; l0 += 2) {
    // two layers' loads in flight before their reductions
    u32x4 f[2][CPL], c[2][CPL];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int l = l0 + j;
#pragma unroll
      for (int k = 0; k < CPL; ++k) {
        const int pc = lane + 64 * k;
        f[j][k] = c[j][k] = u32x4{0u, 0u, 0u, 0u};
        if (l < p.n_layers && pc < pieces) {
          const size_t off = (size_t)row * p.row_bytes + (size_t)pc * 16;
          f[j][k] = *reinterpret_cast<const u32x4 *>(static_cast<const char *>(p.fresh[l]) + off);
          c[j][k] = *reinterpret_cast<const u32x4 *>(static_cast<const char *>(p.cached[l]) + off);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float s = 0.f;
#pragma unroll
      for (int k = 0; k < CPL; ++k) s += sq_diff<BF16>(f[j][k], c[j][k]);
      s = wave_sum(s);
      if (l0 + j < p.n_layers) acc += sqrtf(s);
    }
  }
  if (lane == 0) p.scores[row] = acc / (float)p.n_layers;
}

// Requests up to kSlabKeys tokens are held in registers whole (32 keys per
// lane); longer ones are streamed through 16k-token slabs, reloaded per pass.
constexpr int kSlabKeys = kTopnThreads * 32;

// Exclusive prefix sum over the waves of a wave-uniform value, in wave order;
// also returns the sum over all waves. wsum: kTopnWaves ints of LDS.
__device__ __forceinline__ int wave_scan(int v, int *wsum, int &total) {
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) wsum[wave] = v;
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kTopnWaves; ++w) {
    const int t = wsum[w];
    before += w < wave ? t : 0;
    total += t;
  }
  __syncthreads();  // wsum is reused by the next call
  return before;
}

// Exclusive prefix sum of v over the threads in thread order.
__device__ __forceinline__ int block_scan(int v, int *wsum) {
  const int lane = threadIdx.x & 63;
  int inc = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(inc, off, 64);
    if (lane >= off) inc += t;
  }
  int total;
  const int before = wave_scan(__shfl(inc, 63, 64), wsum, total);
  return before + inc - v;
}

// Number of set bits of m below this lane.
__device__ __forceinline__ int lanes_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((unsigned)(m >> 32), __builtin_amdgcn_mbcnt_lo((unsigned)m, 0u));
}

__device__ __forceinline__ unsigned long long ballot(bool x) { return __builtin_amdgcn_ballot_w64(x); }

// KPL keys per lane; MULTI: a request may span more than one slab.
template <int KPL, bool MULTI>
__global__ __launch_bounds__(kTopnThreads) void select_topn_kernel(const SelectLaunch p) {
  constexpr int kSlab = kTopnThreads * KPL, kWaveSlab = kSlab / kTopnWaves;
  __shared__ int hist[kHistCopies * kHistStride];
  __shared__ int wsum[kTopnWaves];
  __shared__ unsigned s_lo[kTopnWaves], s_hi[kTopnWaves], s_prefix;
  __shared__ int s_remaining, s_top;
  const int b = blockIdx.x;
  const int L = p.req[b].L_d, n = p.req[b].n;
  if (n <= 0 || L <= 0) return;
  const unsigned *key = reinterpret_cast<const unsigned *>(p.scores + p.req[b].doc0);
  int32_t *out = p.idx + p.req[b].imp0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n_slabs = MULTI ? (L + kSlab - 1) / kSlab : 1;

  // slab s: wave w owns keys s*kSlab + w*kWaveSlab + [0, kWaveSlab); its lane
  // holds key j*64 + lane of that range in k[j]
  unsigned k[KPL];
  int slab_base = 0;  // first key of the wave's range in the loaded slab
  int lane_end = 0;   // key j of this lane is a token when j * 64 < lane_end
  auto load = [&](int s) {
    slab_base = s * kSlab + wave * kWaveSlab;
    lane_end = L - slab_base - lane;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const int i = slab_base + j * 64 + lane;
      k[j] = i < L ? key[i] : 0u;
    }
  };
  auto valid = [&](int j) { return j * 64 < lane_end; };

  // ---- bits common to every key: the radix passes start below them ----------
  unsigned lo = 0xffffffffu, hi = 0u;
  for (int s = 0; s < n_slabs; ++s) {
    load(s);
#pragma unroll
    for (int j = 0; j < KPL; ++j)
      if (valid(j)) {
        lo = min(lo, k[j]);
        hi = max(hi, k[j]);
      }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    lo = min(lo, (unsigned)__shfl_xor((int)lo, off, 64));
    hi = max(hi, (unsigned)__shfl_xor((int)hi, off, 64));
  }
  if (lane == 0) {
    s_lo[wave] = lo;
    s_hi[wave] = hi;
  }
  for (int i = threadIdx.x; i < kHistCopies * kHistStride; i += kTopnThreads) hist[i] = 0;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kTopnWaves; ++w) {
    lo = min(lo, s_lo[w]);
    hi = max(hi, s_hi[w]);
  }
  // undecided low bits: keys agree on every bit at or above `top`
  int top = lo == hi ? 0 : 32 - __builtin_clz(lo ^ hi);
  unsigned prefix = lo & (top == 32 ? 0u : ~((1u << top) - 1u));
  int remaining = n;  // keys still to take among those matching prefix above `top`

  // ---- radix select of the n-th highest key, 8 bits per pass -----------------
  while (top > 0) {
    const int w = min(8, top), shift = top - w;
    const unsigned decided = top == 32 ? 0u : ~0u << top;  // bits matched against prefix
    for (int s = 0; s < n_slabs; ++s) {
      if (MULTI) load(s);
#pragma unroll
      for (int j = 0; j < KPL; ++j)
        if (valid(j) && ((k[j] ^ prefix) & decided) == 0u)
          atomicAdd(&hist[(lane & (kHistCopies - 1)) * kHistStride + ((k[j] >> shift) & ((1u << w) - 1u))], 1);
    }
    __syncthreads();
    // digits from the highest down: the selected one holds the remaining-th key
    if (threadIdx.x == 0) s_top = 0;  // every pass ends the loop unless a digit is chosen
    const int d = (1 << w) - 1 - (int)threadIdx.x;
    int h = 0;
    if (d >= 0) {
#pragma unroll 8
      for (int c = 0; c < kHistCopies; ++c) {
        h += hist[c * kHistStride + d];
        hist[c * kHistStride + d] = 0;  // cleared for the next pass
      }
    }
    const int above = block_scan(h, wsum);
    if (d >= 0 && above < remaining && above + h >= remaining) {
      s_prefix = prefix | ((unsigned)d << shift);
      // every key in the digit is taken: no lower bits need deciding
      s_top = above + h == remaining ? 0 : shift;
      s_remaining = above + h == remaining ? 0x7fffffff : remaining - above;
    }
    __syncthreads();
    prefix = s_prefix;
    top = s_top;
    remaining = s_remaining;
  }
  const unsigned T = prefix;  // keep keys above T and the first `remaining` equal to T

  // ---- ordered compaction, slab by slab --------------------------------------
  int out_base = 0, eq_base = 0;  // kept and equal-to-T keys of earlier slabs
  for (int s = 0; s < n_slabs; ++s) {
    if (MULTI) load(s);
    int n_gt = 0, n_eq = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      n_gt += __popcll(ballot(valid(j) && k[j] > T));
      n_eq += __popcll(ballot(valid(j) && k[j] == T));
    }
    int eq_total, kept_total;
    const int eq_before = eq_base + wave_scan(n_eq, wsum, eq_total);
    const int eq_keep = max(0, min(n_eq, remaining - eq_before));
    int pos = out_base + wave_scan(n_gt + eq_keep, wsum, kept_total);
    if (eq_keep == 0) {
      // no key equal to T to take in this wave (the usual case): keep the keys above T
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        const bool keep = valid(j) && k[j] > T;
        const unsigned long long km = ballot(keep);
        if (keep) out[pos + lanes_below(km)] = slab_base + j * 64 + lane;
        pos += __popcll(km);
      }
    } else {
      int eq_seen = 0;
#pragma unroll
      for (int j = 0; j < KPL; ++j) {
        const bool v = valid(j);
        const unsigned long long eq = ballot(v && k[j] == T);
        const bool keep = (v && k[j] > T) || ((eq >> lane & 1ull) && eq_seen + lanes_below(eq) < eq_keep);
        const unsigned long long km = ballot(keep);
        if (keep) out[pos + lanes_below(km)] = slab_base + j * 64 + lane;
        pos += __popcll(km);
        eq_seen += __popcll(eq);
      }
    }
    out_base += kept_total;
    eq_base += eq_total;
  }
}

}  // namespace

hipError_t launch_select_scores(const SelectLaunch &p, bool bf16, hipStream_t st) {
  if (p.rows <= 0) return hipSuccess;
  const int64_t blocks = (p.rows + kScoreThreads / 64 - 1) / (kScoreThreads / 64);
  const int cpl = (p.row_bytes / 16 + 63) / 64;  // row_bytes <= 4096: at most 4
  auto go = [&](auto kern) { kern<<<(unsigned)blocks, kScoreThreads, 0, st>>>(p); };
  if (bf16) {
    if (cpl <= 1) go(select_score_kernel<true, 1>);
    else if (cpl <= 2) go(select_score_kernel<true, 2>);
    else go(select_score_kernel<true, 4>);
  } else {
    if (cpl <= 1) go(select_score_kernel<false, 1>);
    else if (cpl <= 2) go(select_score_kernel<false, 2>);
    else go(select_score_kernel<false, 4>);
  }
  return hipGetLastError();
}

hipError_t launch_select_topn(const SelectLaunch &p, hipStream_t st) {
  if (p.n_req <= 0) return hipSuccess;
  int longest = 0;
  for (int b = 0; b < p.n_req; ++b) longest = std::max(longest, p.req[b].L_d);
  if (longest > kSlabKeys) select_topn_kernel<16, true><<<p.n_req, kTopnThreads, 0, st>>>(p);
  else select_topn_kernel<32, false><<<p.n_req, kTopnThreads, 0, st>>>(p);
  return hipGetLastError();
}

}  // namespace daf
