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
#include "daf_internal.h"

namespace daf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) unsigned char lds_u8;

constexpr int kTM = 128, kTN = 128, kTK = 64;  // workgroup tile
constexpr int kRowB = kTK * 2;                  // bytes per tile row in LDS
constexpr int kTileB = 128 * kRowB;             // bytes per operand tile (16 KiB)
constexpr int kGemmThreads = 256;               // 4 waves, 2 x 2, 64 x 64 each
constexpr int kGroupM = 8;                      // M-tiles per group of the tile order
constexpr int kRsrcWord3 = 0x00020000;          // raw buffer descriptor word 3 (gfx9 family)

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Copy a 128-row x 64-column tile (rows at `base`, row pitch `row_bytes`) into
// LDS; this wave copies rows 32 wave .. 32 wave + 31 (4 instructions of 8 rows).
// Rows at or past `nrec` bytes read as zero.
__device__ __forceinline__ void copy_tile(const unsigned char *base, int nrec, unsigned char *lds, int wave,
                                          const int (&voff)[4]) {
#if defined(__HIP_DEVICE_COMPILE__)
  const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc((void *)base, 0, nrec, kRsrcWord3);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        r, (void __attribute__((address_space(3))) *)((lds_u8 *)lds + (wave * 32 + i * 8) * kRowB), 16, voff[i], 0,
        0, 0);
#endif
}

struct Frag {
  int a[2][4], b[2][4];  // LDS byte offsets: [block][k16 step]
};

// One k step: the 16 MFMAs of this wave on the tiles in (as, bs). All 16
// fragment reads go out first, so that the MFMAs of the first k16 slice run
// while the later reads land.
__device__ __forceinline__ void mma_step(f32x16 (&acc)[2][2], const unsigned char *as, const unsigned char *bs,
                                         const Frag &f) {
  bf16x8 a[4][2], b[4][2];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      a[ks][j] = *reinterpret_cast<const bf16x8 *>(as + f.a[j][ks]);
      b[ks][j] = *reinterpret_cast<const bf16x8 *>(bs + f.b[j][ks]);
    }
#pragma unroll
  for (int ks = 0; ks < 4; ++ks)
    // D^T blocks: rows are output columns (W rows), columns output rows (A rows)
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[ks][nb], a[ks][mb], acc[mb][nb], 0, 0, 0);
  __builtin_amdgcn_sched_group_barrier(0x100, 16, 0);  // the 16 LDS reads
  __builtin_amdgcn_sched_group_barrier(0x008, 16, 0);  // then the 16 MFMAs
}

__device__ __forceinline__ void k_step(f32x16 (&acc)[2][2], const GemmArgs &p, const unsigned char *as,
                                       const unsigned char *bs, unsigned char *an, unsigned char *bn,
                                       const unsigned char *Ab, const unsigned char *Wb, int a_rows_bytes, int kt,
                                       bool prefetch, int wave, const int (&voff)[4], const Frag &f) {
  // this wave's copies of step kt have landed; after the barrier every
  // wave's have, and every wave is done reading the other buffers (step kt-1)
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt and lgkmcnt left at their maxima
  __syncthreads();
  if (prefetch) {
    const int kb = (kt + 1) * kRowB;
    copy_tile(Ab + kb, a_rows_bytes - kb, an, wave, voff);
    copy_tile(Wb + kb, kTN * p.K * 2 - kb, bn, wave, voff);
  }
  mma_step(acc, as, bs, f);
}

__global__ __launch_bounds__(kGemmThreads, 2) void gemm_bf16_kernel(const GemmArgs p) {
  __shared__ __attribute__((aligned(1024))) unsigned char a_lds0[kTileB];
  __shared__ __attribute__((aligned(1024))) unsigned char b_lds0[kTileB];
  __shared__ __attribute__((aligned(1024))) unsigned char a_lds1[kTileB];
  __shared__ __attribute__((aligned(1024))) unsigned char b_lds1[kTileB];

  // ---- which tile ---------------------------------------------------------------
  const int n_tiles = p.tiles_m * p.tiles_n;
  const int per_xcd = (n_tiles + kXcds - 1) / kXcds;
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int t = xcd * per_xcd + slot;
  if (t >= n_tiles) return;
  const int span = kGroupM * p.tiles_n;
  const int first_m = (t / span) * kGroupM;
  const int gsize = min(p.tiles_m - first_m, kGroupM);
  const int tm = first_m + (t % span) % gsize;
  const int tn = (t % span) / gsize;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, l32 = lane & 31, half = lane >> 5;
  const int wm = wave & 1, wn = wave >> 1;
  const int64_t m0 = (int64_t)tm * kTM;
  const int n0 = tn * kTN;
  const int row_bytes = p.K * 2;
  const int rows_valid = (int)min((int64_t)kTM, p.M - m0);
  const unsigned char *Ab = static_cast<const unsigned char *>(p.A) + m0 * row_bytes;
  const unsigned char *Wb = static_cast<const unsigned char *>(p.W) + (int64_t)n0 * row_bytes;
  const int a_rows_bytes = rows_valid * row_bytes;  // A rows past M read as zero

  int voff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = wave * 32 + i * 8 + lane / 8;
    voff[i] = r * row_bytes + (((lane & 7) ^ swz(r)) << 4);
  }
  Frag f;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int ra = wm * 64 + j * 32 + l32, rb = wn * 64 + j * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      f.a[j][ks] = ra * kRowB + (((2 * ks + half) ^ swz(ra)) << 4);
      f.b[j][ks] = rb * kRowB + (((2 * ks + half) ^ swz(rb)) << 4);
    }
  }

  f32x16 acc[2][2];
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) acc[mb][nb] = f32x16{};

  const int KT = p.K / kTK;
  copy_tile(Ab, a_rows_bytes, a_lds0, wave, voff);
  copy_tile(Wb, kTN * row_bytes, b_lds0, wave, voff);
  for (int kt = 0; kt < KT; kt += 2) {
    k_step(acc, p, a_lds0, b_lds0, a_lds1, b_lds1, Ab, Wb, a_rows_bytes, kt, kt + 1 < KT, wave, voff, f);
    if (kt + 1 < KT)
      k_step(acc, p, a_lds1, b_lds1, a_lds0, b_lds0, Ab, Wb, a_rows_bytes, kt + 1, kt + 2 < KT, wave, voff, f);
  }

  // ---- epilogue -------------------------------------------------------------------
  // every wave is done reading the tiles and no copy is in flight: wave w
  // stages its 64 x 64 fp32 block in buffer w (rows of 256 B, 16-byte chunks
  // XOR-swizzled by row)
  __syncthreads();
  unsigned char *stg = wave == 0 ? a_lds0 : wave == 1 ? b_lds0 : wave == 2 ? a_lds1 : b_lds1;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int row = mb * 32 + l32;
        const int c = nb * 8 + 2 * q + half;  // 4-column chunk of the wave's 64 columns
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[mb][nb][4 * q + e];
        *reinterpret_cast<f32x4 *>(stg + row * 256 + ((c ^ (row & 15)) << 4)) = v;
      }
  // each lane then finishes 8 consecutive columns of one row: 8 rows per pass
  const int cg = lane & 7;
  const int n = n0 + wn * 64 + cg * 8;
  float bias[8];
  {
    bf16x8 bv = bf16x8{};
    if (p.bias) bv = *reinterpret_cast<const bf16x8 *>(static_cast<const __bf16 *>(p.bias) + n);
#pragma unroll
    for (int e = 0; e < 8; ++e) bias[e] = (float)bv[e];
  }
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int row = it * 8 + (lane >> 3);
    const int64_t m = m0 + wm * 64 + row;
    const f32x4 v0 = *reinterpret_cast<const f32x4 *>(stg + row * 256 + (((2 * cg) ^ (row & 15)) << 4));
    const f32x4 v1 = *reinterpret_cast<const f32x4 *>(stg + row * 256 + (((2 * cg + 1) ^ (row & 15)) << 4));
    if (m < p.M) {
      float o[8] = {v0[0], v0[1], v0[2], v0[3], v1[0], v1[1], v1[2], v1[3]};
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
}

}  // namespace

hipError_t launch_gemm(const GemmArgs &a, hipStream_t st) {
  GemmArgs p = a;
  p.tiles_m = (int)((p.M + kTM - 1) / kTM);
  p.tiles_n = p.N / kTN;
  const int n_tiles = p.tiles_m * p.tiles_n;
  if (n_tiles <= 0) return hipSuccess;
  const int per_xcd = (n_tiles + kXcds - 1) / kXcds;
  gemm_bf16_kernel<<<dim3(kXcds * per_xcd), dim3(kGemmThreads), 0, st>>>(p);
  return hipGetLastError();
}

}  // namespace daf
