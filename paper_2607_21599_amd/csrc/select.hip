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
// select_topn_kernel: one 1024-thread workgroup per request. Scores are
// non-negative floats, so their bit patterns order like the values: a radix
// select over four 8-bit digits (histograms in LDS) finds the key T of the
// n-th highest score and how many tokens scoring exactly T to keep; one pass
// in index order then keeps every token above T and the first of those equal
// to T, placing each kept index with a block-wide prefix count, so the output
// comes out sorted.
#include "daf_internal.h"

namespace daf {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kScoreThreads = 256;
constexpr int kTopnThreads = 1024;
constexpr int kTopnWaves = kTopnThreads / 64;

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

// Block-wide exclusive prefix count of `flag` in thread order; returns this
// thread's prefix and sets `total`. Uses `wsum` (kTopnWaves ints of LDS).
__device__ __forceinline__ int block_prefix(bool flag, int *wsum, int &total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const unsigned long long bal = __builtin_amdgcn_ballot_w64(flag);
  const unsigned long long below = lane ? (bal & ((1ull << lane) - 1ull)) : 0ull;
  const int in_wave = __popcll(below);
  if (lane == 0) wsum[wave] = __popcll(bal);
  __syncthreads();
  int before = 0;
  total = 0;
#pragma unroll
  for (int w = 0; w < kTopnWaves; ++w) {
    const int v = wsum[w];
    before += w < wave ? v : 0;
    total += v;
  }
  __syncthreads();  // wsum is reused by the next call
  return before + in_wave;
}

__global__ __launch_bounds__(kTopnThreads) void select_topn_kernel(const SelectLaunch p) {
  __shared__ int hist[256];
  __shared__ int wsum[kTopnWaves];
  __shared__ unsigned s_prefix;
  __shared__ int s_remaining;
  const int b = blockIdx.x;
  const int L = p.req[b].L_d, n = p.req[b].n;
  if (n <= 0 || L <= 0) return;
  const unsigned *key = reinterpret_cast<const unsigned *>(p.scores + p.req[b].doc0);
  int32_t *out = p.idx + p.req[b].imp0;

  // ---- radix select: key T of the n-th highest score -------------------------
  unsigned prefix = 0u, mask = 0u;
  int remaining = n;  // how many still to take among keys matching the prefix
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = threadIdx.x; i < 256; i += kTopnThreads) hist[i] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < L; i += kTopnThreads) {
      const unsigned k = key[i];
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int cum = 0, dsel = 0;
      for (int d = 255; d >= 0; --d) {
        if (cum + hist[d] >= remaining) {
          dsel = d;
          break;
        }
        cum += hist[d];
      }
      s_prefix = prefix | ((unsigned)dsel << shift);
      s_remaining = remaining - cum;
    }
    __syncthreads();
    prefix = s_prefix;
    remaining = s_remaining;
    mask |= 255u << shift;
    __syncthreads();
  }
  const unsigned T = prefix;  // tokens above T are all kept, `remaining` of those equal to T

  // ---- keep in index order -------------------------------------------------
  int kept = 0, ties = 0;
  for (int base = 0; base < L; base += kTopnThreads) {
    const int i = base + threadIdx.x;
    const unsigned k = i < L ? key[i] : 0u;
    const bool gt = i < L && k > T;
    const bool eq = i < L && k == T;
    int n_eq;
    const int tie_rank = ties + block_prefix(eq, wsum, n_eq);
    const bool sel = gt || (eq && tie_rank < remaining);
    int n_sel;
    const int pos = kept + block_prefix(sel, wsum, n_sel);
    if (sel) out[pos] = i;
    kept += n_sel;
    ties += n_eq;
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
  select_topn_kernel<<<p.n_req, kTopnThreads, 0, st>>>(p);
  return hipGetLastError();
}

}  // namespace daf
