// Row movement for DAF: the important-row gather (Sec. 2 item 1), the hybrid
// KV write-back and question KV append (Sec. 2 item 2) and the state-fusion
// scatter (Sec. 2 item 3). All are bit copies of whole rows, HBM-bound.
//
// One wave moves one row at a time in 16-byte units (global_load_dwordx4 /
// global_store_dwordx4): consecutive lanes touch consecutive 16 bytes, so
// every row is read and written with fully coalesced 1 KiB wave accesses.
// Each lane issues up to four loads before its stores to keep several
// requests in flight. The row's source/destination index is resolved once per
// row from the request table (kernel argument) and the idx array.
#include "daf_internal.h"

namespace daf {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowThreads = 256;
constexpr int kUnroll = 4;

__device__ __forceinline__ void copy_row(const u32x4 *__restrict__ src, u32x4 *__restrict__ dst,
                                         int units, int lane) {
  for (int u0 = lane; u0 < units; u0 += 64 * kUnroll) {
    u32x4 buf[kUnroll];
#pragma unroll
    for (int j = 0; j < kUnroll; ++j) {
      const int u = u0 + 64 * j;
      if (u < units) buf[j] = __builtin_nontemporal_load(src + u);
    }
#pragma unroll
    for (int j = 0; j < kUnroll; ++j) {
      const int u = u0 + 64 * j;
      if (u < units) __builtin_nontemporal_store(buf[j], dst + u);
    }
  }
}

// request that owns flattened important row r (rows ordered by imp0)
__device__ __forceinline__ int find_imp(const RowLaunch &p, int r) {
  int b = 0;
  while (b + 1 < p.n_req && p.r[b + 1].imp0 - p.r[0].imp0 <= r) ++b;
  return b;
}
__device__ __forceinline__ int find_q(const RowLaunch &p, int j) {
  int b = 0;
  while (b + 1 < p.n_req && p.r[b + 1].q0 - p.r[0].q0 <= j) ++b;
  return b;
}

// dst[imp0 + i] = src[base + idx[imp0 + i]]
__global__ __launch_bounds__(kRowThreads) void gather_rows_kernel(const RowLaunch p,
                                                                   const u32x4 *__restrict__ src,
                                                                   u32x4 *__restrict__ dst) {
  const int lane = threadIdx.x & 63;
  const int waves = gridDim.x * (kRowThreads / 64);
  for (int r = blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6); r < p.total_imp; r += waves) {
    const int b = find_imp(p, r);
    const int e = p.r[0].imp0 + r;  // global important row / idx entry
    const int64_t srow = p.r[b].base + p.idx[e];
    copy_row(src + srow * p.units, dst + (int64_t)e * p.units, p.units, lane);
  }
}

// Important part:  dst[base + idx[imp0 + i]] = src_imp[imp0 + i]
// Question part:   dst[base + L_d + j]       = src_q[q0 + j]
__global__ __launch_bounds__(kRowThreads) void scatter_rows_kernel(const RowLaunch p,
                                                                    ScatterPair a, ScatterPair c,
                                                                    int n_pairs) {
  const int lane = threadIdx.x & 63;
  const int waves = gridDim.x * (kRowThreads / 64);
  const int total = p.total_imp + p.total_q;
  for (int r = blockIdx.x * (kRowThreads / 64) + (threadIdx.x >> 6); r < total; r += waves) {
    int64_t srow, drow;
    bool imp;
    if (r < p.total_imp) {
      const int b = find_imp(p, r);
      const int e = p.r[0].imp0 + r;
      srow = e;
      drow = p.r[b].base + p.idx[e];
      imp = true;
    } else {
      const int j = r - p.total_imp;
      const int b = find_q(p, j);
      const int q = p.r[0].q0 + j;
      srow = q;
      drow = p.r[b].base + p.r[b].L_d + (q - p.r[b].q0);
      imp = false;
    }
    {
      const u32x4 *s = static_cast<const u32x4 *>(imp ? a.src_imp : a.src_q);
      copy_row(s + srow * p.units, static_cast<u32x4 *>(a.dst) + drow * p.units, p.units, lane);
    }
    if (n_pairs > 1) {
      const u32x4 *s = static_cast<const u32x4 *>(imp ? c.src_imp : c.src_q);
      copy_row(s + srow * p.units, static_cast<u32x4 *>(c.dst) + drow * p.units, p.units, lane);
    }
  }
}

// Count idx entries out of [0, L_d) or not above their predecessor. One
// workgroup; the count is reduced in LDS and written (or added) by thread 0.
__global__ __launch_bounds__(1024) void check_indices_kernel(const RowLaunch p, int32_t *bad,
                                                             int accumulate) {
  __shared__ int cnt;
  if (threadIdx.x == 0) cnt = 0;
  __syncthreads();
  int mine = 0;
  for (int r = threadIdx.x; r < p.total_imp; r += blockDim.x) {
    const int b = find_imp(p, r);
    const int e = p.r[0].imp0 + r;
    const int v = p.idx[e];
    bool ok = v >= 0 && v < p.r[b].L_d;
    if (e > p.r[b].imp0) ok = ok && v > p.idx[e - 1];
    mine += ok ? 0 : 1;
  }
  if (mine) atomicAdd(&cnt, mine);
  __syncthreads();
  if (threadIdx.x == 0) *bad = accumulate ? (*bad + cnt) : cnt;
}

int row_grid(int rows) {
  const int blocks = (rows + (kRowThreads / 64) - 1) / (kRowThreads / 64);
  return blocks < 8192 ? (blocks > 0 ? blocks : 1) : 8192;
}

}  // namespace

hipError_t launch_gather(const RowLaunch &p, int64_t, const void *src, void *dst, hipStream_t st) {
  if (p.total_imp <= 0) return hipSuccess;
  gather_rows_kernel<<<row_grid(p.total_imp), kRowThreads, 0, st>>>(
      p, static_cast<const u32x4 *>(src), static_cast<u32x4 *>(dst));
  return hipGetLastError();
}

hipError_t launch_scatter(const RowLaunch &p, const ScatterPair *pairs, int n_pairs, hipStream_t st) {
  const int total = p.total_imp + p.total_q;
  if (total <= 0 || n_pairs <= 0) return hipSuccess;
  scatter_rows_kernel<<<row_grid(total), kRowThreads, 0, st>>>(p, pairs[0],
                                                               n_pairs > 1 ? pairs[1] : pairs[0], n_pairs);
  return hipGetLastError();
}

hipError_t launch_check_indices(const RowLaunch &p, int32_t *d_bad, int accumulate, hipStream_t st) {
  check_indices_kernel<<<1, 1024, 0, st>>>(p, d_bad, accumulate);
  return hipGetLastError();
}

}  // namespace daf
