// Row movement for DAF: the important-row gather (Sec. 2 item 1), the hybrid
// KV write-back and question KV append (Sec. 2 item 2) and the state-fusion
// scatter (Sec. 2 item 3). All are bit copies of whole rows, HBM-bound.
//
// Rows move in 16-byte units (buffer_load_dwordx4 / buffer_store_dwordx4):
// consecutive lanes touch consecutive 16 bytes, so every wave access is a
// fully coalesced 1 KiB. A wave owns a few rows and issues the
// loads of all of them (for both K and V in the KV scatter) before its first
// store, keeping several KiB in flight per wave. A row's source and
// destination are resolved once per row from the request table (a kernel
// argument) and the idx array.
#include "daf_internal.h"

namespace daf {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRowThreads = 256;
constexpr int kRowWaves = kRowThreads / 64;

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

// Raw buffer descriptor over one row (word 3: raw buffer, gfx9 family); loads
// past num_records return zero, stores past it are dropped. The builtins exist
// only for the GPU target, which is the only pass that runs this code.
constexpr int kRsrcWord3 = 0x00020000;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t row_rsrc(const void *base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, bytes, kRsrcWord3);
}
__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, int off) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
#else
  return u32x4{};
#endif
}
__device__ __forceinline__ void store16(__amdgpu_buffer_rsrc_t r, int off, u32x4 v) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, 0);
#endif
}

// Source and destination row of flattened row r of a gather (dst row = the
// global important row) or a scatter (important rows, then question rows).
struct RowMap {
  int64_t src, dst;
  bool imp;
};
__device__ __forceinline__ RowMap gather_map(const RowLaunch &p, int r) {
  const int b = find_imp(p, r);
  const int e = p.r[0].imp0 + r;
  return RowMap{p.r[b].base + p.idx[e], (int64_t)e, true};
}
__device__ __forceinline__ RowMap scatter_map(const RowLaunch &p, int r) {
  if (r < p.total_imp) {
    const int b = find_imp(p, r);
    const int e = p.r[0].imp0 + r;
    return RowMap{(int64_t)e, p.r[b].base + p.idx[e], true};
  }
  const int j = r - p.total_imp;
  const int b = find_q(p, j);
  const int q = p.r[0].q0 + j;
  return RowMap{(int64_t)q, p.r[b].base + p.r[b].L_d + (q - p.r[b].q0), false};
}

// Each wave moves RPW rows of up to 64*UPL 16-byte units for NP tensor pairs:
// every load of all its rows is issued before the first store, so a wave keeps
// RPW*UPL*NP KiB in flight instead of one row's worth. The wave index goes
// through readfirstlane so that row lookups in the request table (a kernel
// argument) compile to scalar loads.
template <int UPL, int RPW, int NP, bool GATHER>
__global__ __launch_bounds__(kRowThreads) void move_rows_kernel(const RowLaunch p, const ScatterPair a,
                                                               const ScatterPair c) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int total = GATHER ? p.total_imp : p.total_imp + p.total_q;
  const int r0 = (blockIdx.x * kRowWaves + wave) * RPW;
  if (r0 >= total) return;
  RowMap m[RPW];
#pragma unroll
  for (int j = 0; j < RPW; ++j)
    if (r0 + j < total) m[j] = GATHER ? gather_map(p, r0 + j) : scatter_map(p, r0 + j);
  // Each row is addressed through a buffer descriptor covering exactly that
  // row: lanes past the row's end load zeros and their stores are dropped by
  // the range check, so the copy has no per-lane branches. Rows wider than
  // 64*UPL units are moved in column chunks.
  const int row_bytes = p.units * 16;
  for (int c0 = 0; c0 < p.units; c0 += 64 * UPL) {
    u32x4 buf[NP][RPW][UPL];
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      if (r0 + j >= total) break;
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        const void *base = m[j].imp ? (q == 0 ? a.src_imp : c.src_imp) : (q == 0 ? a.src_q : c.src_q);
        const auto rs = row_rsrc(static_cast<const char *>(base) + m[j].src * row_bytes, row_bytes);
#pragma unroll
        for (int k = 0; k < UPL; ++k) buf[q][j][k] = load16(rs, (c0 + lane + 64 * k) * 16);
      }
    }
#pragma unroll
    for (int j = 0; j < RPW; ++j) {
      if (r0 + j >= total) break;
#pragma unroll
      for (int q = 0; q < NP; ++q) {
        const auto rd = row_rsrc(static_cast<char *>(q == 0 ? a.dst : c.dst) + m[j].dst * row_bytes, row_bytes);
#pragma unroll
        for (int k = 0; k < UPL; ++k) store16(rd, (c0 + lane + 64 * k) * 16, buf[q][j][k]);
      }
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

// Launch with UPL = units per lane per row (rounded up to one of 1, 2, 4, 8;
// wider rows go in chunks of 8) and rows per wave for about 8 KiB in flight
// per wave and tensor.
template <int NP, bool GATHER>
hipError_t launch_move(const RowLaunch &p, const ScatterPair &a, const ScatterPair &c, int rows, hipStream_t st) {
  const int upl = (p.units + 63) / 64;
  auto go = [&](auto kern, int rpw) {
    const int waves = (rows + rpw - 1) / rpw;
    kern<<<(waves + kRowWaves - 1) / kRowWaves, kRowThreads, 0, st>>>(p, a, c);
  };
  // several rows per wave only when there are enough rows to keep every CU
  // busy with ~32 waves anyway; otherwise one row per wave (the index load
  // of each row is a serial latency the other waves hide)
  const bool many = rows >= 256 * 32 * 4;
  if (upl <= 1) many ? go(move_rows_kernel<1, 4, NP, GATHER>, 4) : go(move_rows_kernel<1, 1, NP, GATHER>, 1);
  else if (upl <= 2) many ? go(move_rows_kernel<2, 2, NP, GATHER>, 2) : go(move_rows_kernel<2, 1, NP, GATHER>, 1);
  else if (upl <= 4) go(move_rows_kernel<4, 1, NP, GATHER>, 1);
  else go(move_rows_kernel<8, 1, NP, GATHER>, 1);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gather(const RowLaunch &p, int64_t, const void *src, void *dst, hipStream_t st) {
  if (p.total_imp <= 0) return hipSuccess;
  const ScatterPair a{src, src, dst};
  return launch_move<1, true>(p, a, a, p.total_imp, st);
}

hipError_t launch_scatter(const RowLaunch &p, const ScatterPair *pairs, int n_pairs, hipStream_t st) {
  const int total = p.total_imp + p.total_q;
  if (total <= 0 || n_pairs <= 0) return hipSuccess;
  if (n_pairs > 1) return launch_move<2, false>(p, pairs[0], pairs[1], total, st);
  return launch_move<1, false>(p, pairs[0], pairs[0], total, st);
}

hipError_t launch_check_indices(const RowLaunch &p, int32_t *d_bad, int accumulate, hipStream_t st) {
  check_indices_kernel<<<1, 1024, 0, st>>>(p, d_bad, accumulate);
  return hipGetLastError();
}

}  // namespace daf
