// Dense bf16 projections around the DAF attention: C = A W^T (+ bias)
// (+ residual), A [M][K] and W [N][K] row-major, fp32 accumulation, bf16 out.
// These are the QKV, output and MLP projections of a decoder layer, which the
// paper's layer runs on the important and question rows only (Sec. 2 item 2:
// the QKV computation phase; Sec. 2 item 3: the fused compact state feeds the
// next layer's projections).
//
// Both operands are K-contiguous, which is how the matrix cores take them: a
// 32x32x16 bf16 MFMA reads, per lane, 8 consecutive k of one row of each
// operand. Workgroup tile 128 (M) x 128 (N), k steps of 64; 4 waves of 64 x 64
// (2 x 2 MFMA blocks). The A and W tiles of a k step are copied global -> LDS
// with the buffer unit (rows of 128 B, 16-byte chunks XOR-swizzled by
// (row >> 1) & 7 so that the 16 lanes of a read phase hit distinct banks),
// double-buffered so the copy of step k+1 overlaps the MFMAs of step k. The
// accumulators are staged through LDS in fp32 so that bias, residual and the
// bf16 stores run on whole 128-byte row segments.
//
// Tile order: the tiles are split into 8 contiguous ranges, one per XCD
// (workgroup i runs on XCD i mod 8); within a range, groups of 8 M-tiles sweep
// the N-tiles, so the A rows of a group stay in that XCD's L2 while W streams.
#include <algorithm>

#include "daf_internal.h"

namespace daf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) unsigned char lds_u8;

constexpr int kTK = 64;                         // k step
constexpr int kRowB = kTK * 2;                  // bytes per tile row in LDS
constexpr int kGroupM = 8;                      // M-tiles per group of the tile order
[[maybe_unused]] constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Tile shape: workgroup TM x TN, waves of WM x WN (TM/WM x TN/WN waves).
template <int TM_, int TN_, int WM_, int WN_>
struct Shape {
  static constexpr int TM = TM_, TN = TN_, WM = WM_, WN = WN_;
  static constexpr int WAVES_M = TM / WM, WAVES = WAVES_M * (TN / WN), THREADS = 64 * WAVES;
  static constexpr int MB = WM / 32, NB = WN / 32;           // 32x32 MFMA blocks per wave
  static constexpr int A_IPW = TM / WAVES / 8, B_IPW = TN / WAVES / 8;  // copy instructions per wave
  static constexpr int ATILE = TM * kRowB, BTILE = TN * kRowB;
  // fp32 staging of the epilogue: rows per pass so that a wave's share fits
  // its part of the LDS (2 (ATILE + BTILE) / WAVES bytes, 256 B per row)
  static constexpr int STAGE_B = 2 * (ATILE + BTILE) / WAVES;
  static constexpr int PASS_ROWS = (STAGE_B / (WN * 4)) < WM ? (STAGE_B / (WN * 4)) : WM;
  static_assert(WN == 64, "the epilogue stages 64-column rows");
  static_assert(TM % (WAVES * 8) == 0 && TN % (WAVES * 8) == 0, "copy split");
  static_assert(WM % PASS_ROWS == 0 && PASS_ROWS % 8 == 0, "staging passes");
};

// Copy ROWS rows x 64 columns (rows at `base`, pitch `row_bytes`) into LDS;
// this wave copies IPW x 8 rows starting at row first_row. Rows at or past
// `nrec` bytes read as zero.
template <int IPW>
__device__ __forceinline__ void copy_tile(const unsigned char *base, int nrec, unsigned char *lds, int first_row,
                                          const int (&voff)[IPW]) {
#if defined(__HIP_DEVICE_COMPILE__)
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, nrec, kRsrcWord3);
#pragma unroll
  for (int i = 0; i < IPW; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        r, (void __attribute__((address_space(3))) *)((lds_u8 *)lds + (first_row + i * 8) * kRowB), 16, voff[i], 0,
        0, 0);
#endif
}

// One k step: the MB x NB x 4 MFMAs of this wave on the tiles in (as, bs).
// The fragment reads of each half of the step (two k16 slices) go out before
// its MFMAs, so the MFMAs of one slice run while the next reads land.
template <class S>
__device__ __forceinline__ void mma_step(f32x16 (&acc)[S::MB][S::NB], const unsigned char *as,
                                         const unsigned char *bs, const int (&fa)[S::MB][4],
                                         const int (&fb)[S::NB][4]) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    bf16x8 a[2][S::MB], b[2][S::NB];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int j = 0; j < S::MB; ++j) a[kk][j] = *reinterpret_cast<const bf16x8 *>(as + fa[j][2 * h + kk]);
#pragma unroll
      for (int j = 0; j < S::NB; ++j) b[kk][j] = *reinterpret_cast<const bf16x8 *>(bs + fb[j][2 * h + kk]);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
      // D^T blocks: rows are output columns (W rows), columns output rows (A rows)
#pragma unroll
      for (int mb = 0; mb < S::MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < S::NB; ++nb)
          acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[kk][nb], a[kk][mb], acc[mb][nb], 0, 0, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * (S::MB + S::NB), 0);  // this half's LDS reads
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * S::MB * S::NB, 0);    // then its MFMAs
  }
}

template <class S>
__device__ __forceinline__ void k_step(f32x16 (&acc)[S::MB][S::NB], int b_rows_bytes, const unsigned char *as,
                                       const unsigned char *bs, unsigned char *an, unsigned char *bn,
                                       const unsigned char *Ab, const unsigned char *Wb, int a_rows_bytes, int kt,
                                       bool prefetch, int wave, const int (&va)[S::A_IPW],
                                       const int (&vb)[S::B_IPW], const int (&fa)[S::MB][4],
                                       const int (&fb)[S::NB][4]) {
  // this wave's copies of step kt have landed; after the barrier every
  // wave's have, and every wave is done reading the other buffers (step kt-1)
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt and lgkmcnt left at their maxima
  __syncthreads();
  if (prefetch) {
    const int kb = (kt + 1) * kRowB;
    copy_tile<S::A_IPW>(Ab + kb, a_rows_bytes - kb, an, wave * S::A_IPW * 8, va);
    copy_tile<S::B_IPW>(Wb + kb, b_rows_bytes - kb, bn, wave * S::B_IPW * 8, vb);
  }
  mma_step<S>(acc, as, bs, fa, fb);
}

// Output tile t of the tile order: groups of kGroupM M-tiles sweep the N-tiles.
__device__ __forceinline__ void tile_coords(const GemmArgs &p, int t, int &tm, int &tn) {
  const int span = kGroupM * p.tiles_n;
  const int first_m = (t / span) * kGroupM;
  const int gsize = min(p.tiles_m - first_m, kGroupM);
  tm = first_m + (t % span) % gsize;
  tn = (t % span) / gsize;
}

// GLU: the tile's TN W rows are TN/2 gate rows and the matching TN/2 up rows
// (N rows further), so the workgroup produces TN/2 gated output columns.
// PARTIAL: one k piece of a tail tile, its fp32 sums stored to p.part.
template <class S, bool GLU, bool PARTIAL = false>
__global__ __launch_bounds__(S::THREADS, 2) void gemm_bf16_kernel(const GemmArgs p) {
  __shared__ __attribute__((aligned(1024))) unsigned char a_lds0[S::ATILE];
  __shared__ __attribute__((aligned(1024))) unsigned char b_lds0[S::BTILE];
  __shared__ __attribute__((aligned(1024))) unsigned char a_lds1[S::ATILE];
  __shared__ __attribute__((aligned(1024))) unsigned char b_lds1[S::BTILE];

  // ---- which tile ---------------------------------------------------------------
  // whole tiles: the launch's range of the tile order is cut into 8 contiguous
  // ranges, one per XCD (workgroup i runs on XCD i mod 8); k pieces of tail
  // tiles: workgroup i runs piece i mod k_parts of tile t_begin + i / k_parts
  int t, kp = 0;
  if (PARTIAL) {
    if ((int)blockIdx.x >= p.t_count * p.k_parts) return;
    t = p.t_begin + blockIdx.x / p.k_parts;
    kp = blockIdx.x % p.k_parts;
  } else {
    const int count = p.t_count > 0 ? p.t_count : p.tiles_m * p.tiles_n;
    const int per_xcd = (count + kXcds - 1) / kXcds;
    const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
    if (xcd * per_xcd + slot >= count) return;
    t = p.t_begin + xcd * per_xcd + slot;
  }
  int tm, tn;
  tile_coords(p, t, tm, tn);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l32 = lane & 31, half = lane >> 5;
  const int wm = wave % S::WAVES_M, wn = wave / S::WAVES_M;
  const int64_t m0 = (int64_t)tm * S::TM;
  constexpr int OUT_TN = GLU ? S::TN / 2 : S::TN;  // output columns per tile
  const int n0 = tn * OUT_TN;
  const int row_bytes = p.K * 2;
  const int rows_valid = (int)min((int64_t)S::TM, p.M - m0);
  const unsigned char *Ab = static_cast<const unsigned char *>(p.A) + m0 * row_bytes;
  const unsigned char *Wb = static_cast<const unsigned char *>(p.W) + (int64_t)n0 * row_bytes;
  const int a_rows_bytes = rows_valid * row_bytes;  // A rows past M read as zero
  // W rows the tile reaches from Wb: TN, or up to the last up row in GLU mode
  const int b_rows_bytes = (GLU ? p.N + S::TN / 2 : S::TN) * row_bytes;

  int va[S::A_IPW], vb[S::B_IPW];
#pragma unroll
  for (int i = 0; i < S::A_IPW; ++i) {
    const int r = (wave * S::A_IPW + i) * 8 + lane / 8;
    va[i] = r * row_bytes + (((lane & 7) ^ swz(r)) << 4);
  }
#pragma unroll
  for (int i = 0; i < S::B_IPW; ++i) {
    const int r = (wave * S::B_IPW + i) * 8 + lane / 8;
    const int g = GLU && r >= S::TN / 2 ? p.N + r - S::TN / 2 : r;  // W row relative to Wb
    vb[i] = g * row_bytes + (((lane & 7) ^ swz(r)) << 4);
  }
  int fa[S::MB][4], fb[S::NB][4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
    for (int j = 0; j < S::MB; ++j) {
      const int ra = wm * S::WM + j * 32 + l32;
      fa[j][ks] = ra * kRowB + (((2 * ks + half) ^ swz(ra)) << 4);
    }
#pragma unroll
    for (int j = 0; j < S::NB; ++j) {
      const int rb = wn * S::WN + j * 32 + l32;
      fb[j][ks] = rb * kRowB + (((2 * ks + half) ^ swz(rb)) << 4);
    }
  }

  f32x16 acc[S::MB][S::NB];
#pragma unroll
  for (int mb = 0; mb < S::MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < S::NB; ++nb) acc[mb][nb] = f32x16{};

  const int KT = p.K / kTK;
  const int kt0 = PARTIAL ? kp * KT / p.k_parts : 0, kt1 = PARTIAL ? (kp + 1) * KT / p.k_parts : KT;
  copy_tile<S::A_IPW>(Ab + kt0 * kRowB, a_rows_bytes - kt0 * kRowB, a_lds0, wave * S::A_IPW * 8, va);
  copy_tile<S::B_IPW>(Wb + kt0 * kRowB, b_rows_bytes - kt0 * kRowB, b_lds0, wave * S::B_IPW * 8, vb);
  for (int kt = kt0; kt < kt1; kt += 2) {
    k_step<S>(acc, b_rows_bytes, a_lds0, b_lds0, a_lds1, b_lds1, Ab, Wb, a_rows_bytes, kt, kt + 1 < kt1, wave, va,
              vb, fa, fb);
    if (kt + 1 < kt1)
      k_step<S>(acc, b_rows_bytes, a_lds1, b_lds1, a_lds0, b_lds0, Ab, Wb, a_rows_bytes, kt + 1, kt + 2 < kt1, wave,
                va, vb, fa, fb);
  }

  // ---- epilogue -------------------------------------------------------------------
  // every wave is done reading the tiles and no copy is in flight: the four
  // tile buffers become staging space, STAGE_B bytes per wave (fp32 rows of
  // 256 B, 16-byte chunks XOR-swizzled by row), PASS_ROWS rows per pass
  __syncthreads();
  // wave w's region: bytes [w STAGE_B, (w+1) STAGE_B) of a_lds0 | b_lds0 |
  // a_lds1 | b_lds1 taken in this order (a region never straddles two)
  auto stage_of = [&](int w) -> unsigned char * {
    const int off = w * S::STAGE_B;
    constexpr int A = S::ATILE, B = S::BTILE;
    return off < A ? a_lds0 + off : off < A + B ? b_lds0 + (off - A) : off < 2 * A + B ? a_lds1 + (off - A - B)
                                                                                       : b_lds1 + (off - 2 * A - B);
  };
  unsigned char *stg = stage_of(wave);
  constexpr int WAVES_N = S::TN / S::WN;
  // GLU: the gate waves (wn < WAVES_N / 2) finish the rows; their partner
  // holds the up block of the same output columns
  const bool finisher = !GLU || wn < WAVES_N / 2;
  const unsigned char *stg_up = GLU ? stage_of(wave + S::WAVES_M * (WAVES_N / 2)) : stg;
  const int cg = lane & 7;
  const int n = n0 + wn * S::WN + cg * 8;
  float bias[8];
  {
    bf16x8 bv = bf16x8{};
    if (!GLU && !PARTIAL && p.bias) bv = *reinterpret_cast<const bf16x8 *>(static_cast<const __bf16 *>(p.bias) + n);
#pragma unroll
    for (int e = 0; e < 8; ++e) bias[e] = (float)bv[e];
  }
#pragma unroll
  for (int pass = 0; pass < S::WM / S::PASS_ROWS; ++pass) {
#pragma unroll
    for (int mb = 0; mb < S::MB; ++mb) {
      if (mb * 32 / S::PASS_ROWS != pass && S::PASS_ROWS >= 32) continue;
#pragma unroll
      for (int nb = 0; nb < S::NB; ++nb)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int row = mb * 32 + l32 - pass * S::PASS_ROWS;
          const int c = nb * 8 + 2 * q + half;  // 4-column chunk of the wave's 64 columns
          f32x4 v;
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[mb][nb][4 * q + e];
          *reinterpret_cast<f32x4 *>(stg + row * 256 + ((c ^ (row & 15)) << 4)) = v;
        }
    }
    if (GLU) __syncthreads();  // the partner's up block is staged
    // each lane then finishes 8 consecutive columns of one row: 8 rows per round
#pragma unroll
    for (int it = 0; it < S::PASS_ROWS / 8; ++it) {
      if (!finisher) break;
      const int row = it * 8 + (lane >> 3);
      const int64_t m = m0 + wm * S::WM + pass * S::PASS_ROWS + row;
      const f32x4 v0 = *reinterpret_cast<const f32x4 *>(stg + row * 256 + (((2 * cg) ^ (row & 15)) << 4));
      const f32x4 v1 = *reinterpret_cast<const f32x4 *>(stg + row * 256 + (((2 * cg + 1) ^ (row & 15)) << 4));
      if (PARTIAL) {
        // the piece's fp32 sums: [TM][TN] per (tail tile, piece)
        if (m < p.M) {
          float *dst = p.part + ((size_t)(t - p.t_begin) * p.k_parts + kp) * (S::TM * S::TN) +
                       (size_t)(m - m0) * S::TN + (n - n0);
          *reinterpret_cast<f32x4 *>(dst) = v0;
          *reinterpret_cast<f32x4 *>(dst + 4) = v1;
        }
        continue;
      }
      if (m < p.M) {
        float o[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
        if (GLU) {
          const f32x4 u0 = *reinterpret_cast<const f32x4 *>(stg_up + row * 256 + (((2 * cg) ^ (row & 15)) << 4));
          const f32x4 u1 =
              *reinterpret_cast<const f32x4 *>(stg_up + row * 256 + (((2 * cg + 1) ^ (row & 15)) << 4));
          const float u[8] = {u0[0], u0[1], u0[2], u0[3], u1[0], u1[1], u1[2], u1[3]};
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = o[e] / (1.0f + __expf(-o[e])) * u[e];
        }
        if (p.residual) {
          const bf16x8 rv = *reinterpret_cast<const bf16x8 *>(static_cast<const __bf16 *>(p.residual) + m * p.N + n);
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] += (float)rv[e];
        }
        bf16x8 out;
#pragma unroll
        for (int e = 0; e < 8; ++e) out[e] = (__bf16)(o[e] + bias[e]);
        *reinterpret_cast<bf16x8 *>(static_cast<__bf16 *>(p.C) + m * p.N + n) = out;
      }
    }
    if (GLU) __syncthreads();  // the next pass restages over these rows
  }
}

// The tail tiles' k pieces summed: C = sum of pieces (+ residual) (+ bias), in
// the order of the whole-tile epilogue. One thread per 8 columns of a row.
template <class S>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(const GemmArgs p) {
  constexpr int CHUNKS = S::TN / 8;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t per_tile = (int64_t)S::TM * CHUNKS;
  if (gid >= per_tile * p.t_count) return;
  const int tl = (int)(gid / per_tile);
  const int row = (int)(gid % per_tile) / CHUNKS, cg = (int)(gid % per_tile) % CHUNKS;
  int tm, tn;
  tile_coords(p, p.t_begin + tl, tm, tn);
  const int64_t m = (int64_t)tm * S::TM + row;
  if (m >= p.M) return;
  const int n = tn * S::TN + cg * 8;
  float o[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const float *src = p.part + (size_t)tl * p.k_parts * (S::TM * S::TN) + (size_t)row * S::TN + cg * 8;
  for (int k = 0; k < p.k_parts; ++k) {
    const f32x4 a = *reinterpret_cast<const f32x4 *>(src + (size_t)k * (S::TM * S::TN));
    const f32x4 b = *reinterpret_cast<const f32x4 *>(src + (size_t)k * (S::TM * S::TN) + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] += a[e];
      o[4 + e] += b[e];
    }
  }
  if (p.residual) {
    const bf16x8 rv = *reinterpret_cast<const bf16x8 *>(static_cast<const __bf16 *>(p.residual) + m * p.N + n);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] += (float)rv[e];
  }
  bf16x8 bv = bf16x8{};
  if (p.bias) bv = *reinterpret_cast<const bf16x8 *>(static_cast<const __bf16 *>(p.bias) + n);
  bf16x8 out;
#pragma unroll
  for (int e = 0; e < 8; ++e) out[e] = (__bf16)(o[e] + (float)bv[e]);
  *reinterpret_cast<bf16x8 *>(static_cast<__bf16 *>(p.C) + m * p.N + n) = out;
}

using SmallTile = Shape<128, 128, 64, 64>;  // 4 waves, two workgroups per CU
using LargeTile = Shape<256, 256, 128, 64>;  // 8 waves, one workgroup per CU

template <class S>
hipError_t launch_shape(GemmArgs p, hipStream_t st) {
  p.tiles_m = (int)((p.M + S::TM - 1) / S::TM);
  p.tiles_n = p.N / (p.glu ? S::TN / 2 : S::TN);
  const int n_tiles = p.tiles_m * p.tiles_n;
  if (n_tiles <= 0) return hipSuccess;
  const int per_xcd = (n_tiles + kXcds - 1) / kXcds;
  if (p.glu) gemm_bf16_kernel<S, true><<<dim3(kXcds * per_xcd), dim3(S::THREADS), 0, st>>>(p);
  else gemm_bf16_kernel<S, false><<<dim3(kXcds * per_xcd), dim3(S::THREADS), 0, st>>>(p);
  return hipGetLastError();
}

// Whole rounds of the resident workgroups as whole tiles, the remaining tiles
// cut along k into pieces that fill the idle slots, then the reduction.
template <class S>
hipError_t launch_split(GemmArgs p, float *part, size_t part_bytes, hipStream_t st) {
  constexpr int slots = S::THREADS == 256 ? 512 : 256;  // resident workgroups: 2 per CU for 4 waves, else 1
  p.tiles_m = (int)((p.M + S::TM - 1) / S::TM);
  p.tiles_n = p.N / S::TN;
  const int n_tiles = p.tiles_m * p.tiles_n;
  const int full = n_tiles / slots * slots, tail = n_tiles - full;
  const int KT = p.K / kTK;
  const int k_parts = tail > 0 ? std::min(std::min(slots / tail, KT / 4), 8) : 0;
  if (n_tiles <= 0 || k_parts < 2 || (size_t)tail * k_parts * S::TM * S::TN * 4 > part_bytes)
    return launch_shape<S>(p, st);
  if (full > 0) {
    GemmArgs a = p;
    a.t_begin = 0;
    a.t_count = full;
    gemm_bf16_kernel<S, false><<<dim3(kXcds * ((full + kXcds - 1) / kXcds)), dim3(S::THREADS), 0, st>>>(a);
  }
  GemmArgs b = p;
  b.t_begin = full;
  b.t_count = tail;
  b.k_parts = k_parts;
  b.part = part;
  gemm_bf16_kernel<S, false, true><<<dim3(tail * k_parts), dim3(S::THREADS), 0, st>>>(b);
  const int64_t threads = (int64_t)tail * S::TM * (S::TN / 8);
  gemm_reduce_kernel<S><<<dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, st>>>(b);
  return hipGetLastError();
}

bool use_large(const GemmArgs &a) {
  // the large tile needs whole output tiles (256 columns, 128 gated) and
  // enough tiles to fill the CUs
  const int out_tn = a.glu ? LargeTile::TN / 2 : LargeTile::TN;
  const int64_t large_tiles = ((a.M + LargeTile::TM - 1) / LargeTile::TM) * (a.N / out_tn);
  return a.N % out_tn == 0 && large_tiles >= 2 * 256;
}

}  // namespace

hipError_t launch_gemm_split(const GemmArgs &a, float *part, size_t part_bytes, hipStream_t st) {
  if (a.glu || part == nullptr) return launch_gemm(a, st);
  return use_large(a) ? launch_split<LargeTile>(a, part, part_bytes, st)
                      : launch_split<SmallTile>(a, part, part_bytes, st);
}

hipError_t launch_gemm(const GemmArgs &a, hipStream_t st) {
  return use_large(a) ? launch_shape<LargeTile>(a, st) : launch_shape<SmallTile>(a, st);
}

}  // namespace daf
