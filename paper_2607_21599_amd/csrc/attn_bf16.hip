// bf16 causal GQA flash attention for both DAF attention stages (gfx950).
//
// Same operation and work decomposition as the fp32 kernel in attn.hip (see
// there): query row i of a request sees keys 0 .. i + (n_keys - n_rows), a
// workgroup of 4 waves owns 128 query rows of one head and one key split, and
// the G heads that share a KV head form an XCD-local work group.
//
// bf16 data path, per 64-key tile:
//  * K and V tiles are copied global -> LDS by the buffer unit
//    (buffer_load_dwordx4 ... lds): no VGPR staging, no VALU address math in
//    the loop, and rows past the end of the request read as zeros through the
//    buffer range check. Each 1 KiB DMA instruction writes 1024/(2D) whole rows;
//    16-byte chunks are XOR-swizzled within a row so that the two LDS read
//    patterns below are free of bank conflicts. Two tile buffers: the DMA of
//    tile t+1 runs while tile t is consumed, one barrier per tile.
//  * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (keys on M, query rows on N, Q in
//    registers), so each lane owns one query row.
//  * O^T += V^T P^T: P^T comes straight from the S^T accumulators; the V^T
//    operand (8 consecutive keys of one feature per lane) is read from the
//    row-major V tile with ds_read_b64_tr_b16, which transposes 16-bit data
//    across each 16-lane group.
//  * Online softmax in fp32, base 2, scale folded into one FMA per score. Full
//    tiles form each 32-key half's probabilities against the running max as it
//    stands, without taking the half's max: only when some lane's share of the
//    half's sum exceeds 2^32 (or is not finite, as on a row's first tile) is
//    the half's exact max taken, the running max raised, O and the sum rescaled
//    and the half formed again. Probabilities thus stay below 2^32 (far from
//    overflow in fp32 and bf16) and the S MFMAs of half 1 run beside the
//    softmax of half 0. Diagonal tiles take one max over the tile and raise the
//    running max only when it grows by more than 2^8. The row max of a lane
//    pair is exchanged with v_permlane32_swap.
//  * The row sum is taken from the bf16-rounded probabilities that the P.V
//    product uses (v_dot2c_f32_bf16 against (1, 1), one instruction per pair).
//  * Launch shape for causal self attention: the heaviest 128 jobs of an XCD
//    (one query head of one 128-row block each) are run by its 64 resident
//    workgroups in pairs, job u with job 127 - u, so each workgroup gets a heavy
//    and a light block of near-equal total; lighter jobs get a workgroup each.
#include <math.h>

#include <algorithm>

#include "daf_internal.h"

namespace daf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) unsigned char lds_u8;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr int kBN = 64;                  // keys per tile
[[maybe_unused]] constexpr int kRsrcWord3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)
constexpr float kRescaleSlack = 8.0f;    // log2 units a row max may grow before O is rescaled
// Full tiles skip the max: a half's probabilities are formed with the running
// max as it stands, and only if some lane's share of the half's sum exceeds
// this (or is not finite) is the half's exact max taken, the running max
// raised and the half formed again. Each probability is then at most 2^32, far
// from fp32 and bf16 overflow in the row sum and the O accumulators.
constexpr float kHalfSumLimit = 4294967296.0f;

template <int D>
struct Geo {
  static constexpr int ROWB = D * 2;         // bytes per K/V row in LDS
  static constexpr int CH = D / 8;           // 16-byte chunks per row
  static constexpr int TILE = kBN * ROWB;    // bytes of one K or V tile
  static constexpr int RPI = 64 / CH;        // rows written by one 1 KiB DMA instruction
  static constexpr int IPW = kBN / RPI / 4;  // DMA instructions per wave, per tensor and tile
  static constexpr int DS = D / 16;          // contraction steps of S^T
  static constexpr int DB = D / 32;          // 32-feature output blocks
  static_assert(RPI * ROWB == 1024, "one DMA instruction writes 1 KiB");
};

// chunk swizzles (XOR, so their own inverse), both < CH
__device__ __forceinline__ int swz_k(int r, int ch) { return r & (ch - 1); }
__device__ __forceinline__ int swz_v(int r, int ch) { return (((r & 3) << 2) | ((r >> 2) & 3)) & (ch - 1); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// x and the same register of lane ^ 32: v_permlane32_swap on two copies of x
// leaves {x[l % 32], x[l % 32 + 32]} in the two results. Each result element
// is copied to a scalar before the bit cast (a bit cast of a vector element
// expression reads the vector's first element).
__device__ __forceinline__ void lane_pair(float x, float &a, float &b) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const unsigned r0 = r[0], r1 = r[1];
  a = __builtin_bit_cast(float, r0);
  b = __builtin_bit_cast(float, r1);
}
__device__ __forceinline__ float pair_max(float x) {
  float a, b;
  lane_pair(x, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float pair_sum(float x) {
  float a, b;
  lane_pair(x, a, b);
  return a + b;
}

__device__ __forceinline__ bf16x8 tr_pair(const unsigned char *lds_base, int off_a, int off_b) {
  const lds_u8 *b = (const lds_u8 *)lds_base;
  const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(b + off_a));
  const bf16x4 c = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4 *)(b + off_b));
  return bf16x8{a[0], a[1], a[2], a[3], c[0], c[1], c[2], c[3]};
}

// Copy one 64-key K tile and V tile global -> LDS with the buffer unit. Each
// wave writes its IPW KiB of each tile; rows at or past n_keys read as zero.
template <int IPW>
__device__ __forceinline__ void dma_tile(const unsigned char *kg, const unsigned char *vg, int kb, int n_keys,
                                         int kv_row_bytes, unsigned char *k_lds, unsigned char *v_lds, int wave,
                                         const int (&dma_k)[IPW], const int (&dma_v)[IPW]) {
  // The buffer->LDS builtin only exists for the GPU target; the host pass of
  // this translation unit only needs the kernel's launch stub.
#if defined(__HIP_DEVICE_COMPILE__)
  const int nrec = (n_keys - kb) * kv_row_bytes;
  const __amdgpu_buffer_rsrc_t rk =
      __builtin_amdgcn_make_buffer_rsrc((void *)(kg + (size_t)kb * kv_row_bytes), 0, nrec, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t rv =
      __builtin_amdgcn_make_buffer_rsrc((void *)(vg + (size_t)kb * kv_row_bytes), 0, nrec, kRsrcWord3);
  lds_u8 *kbase = (lds_u8 *)k_lds + wave * IPW * 1024;
  lds_u8 *vbase = (lds_u8 *)v_lds + wave * IPW * 1024;
#pragma unroll
  for (int i = 0; i < IPW; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (void __attribute__((address_space(3))) *)(kbase + i * 1024), 16,
                                             dma_k[i], 0, 0, 0);
#pragma unroll
  for (int i = 0; i < IPW; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (void __attribute__((address_space(3))) *)(vbase + i * 1024), 16,
                                             dma_v[i], 0, 0, 0);
#endif
}

// Output staging: 32 rows of ROWB bytes per wave in LDS, the 16-byte chunks of
// a row XOR-swizzled by the row so that both the per-lane writes (pieces of
// every chunk of one row) and the row-contiguous reads spread over the banks.
// stage_put writes v (8 or 16 bytes) at byte `sub` of logical chunk c of row r.
template <int D, typename V>
__device__ __forceinline__ void stage_put(unsigned char *stg, int r, int c, int sub, const V &v) {
  constexpr int CH = Geo<D>::CH;
  *reinterpret_cast<V *>(stg + r * Geo<D>::ROWB + ((c ^ (r & (CH - 1))) << 4) + sub) = v;
}
// Write the wave's staged rows wrow .. wrow+31 (those below n_rows): each lane
// moves one 16-byte chunk, CH lanes cover a row, so every store instruction
// writes 64/CH whole rows. dst(r) is the byte address of row r's first chunk.
template <int D, typename F>
__device__ __forceinline__ void store_rows(const unsigned char *stg, int lane, int wrow, int n_rows, F dst) {
  constexpr int CH = Geo<D>::CH, RPL = 64 / CH;
  const int j = lane % CH;
#pragma unroll
  for (int it = 0; it < 32 / RPL; ++it) {
    const int r = it * RPL + lane / CH;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(stg + r * Geo<D>::ROWB + ((j ^ (r & (CH - 1))) << 4));
    if (wrow + r < n_rows) *reinterpret_cast<u32x4 *>(dst(wrow + r) + j * 16) = v;
  }
}

// Per-wave state of one workgroup tile (lives in registers after inlining).
template <int D>
struct WaveState {
  using Gm = Geo<D>;
  bf16x8 qf[Gm::DS];       // Q rows as the B operand of S^T
  f32x16 oacc[Gm::DB];     // O^T accumulators
  float m_run;             // running max, scaled base-2 units, equal in both halves
  float l_run;             // this lane's share of the row sum
  int koff[Gm::DS];        // K tile read offsets
  int voff[Gm::DB][2];     // V tile transposed-read offsets
  int dma_k[Gm::IPW], dma_v[Gm::IPW];
  const unsigned char *kg, *vg;
  int n_keys, kv_row_bytes, limit, half, wave;
  int wave_last_key;       // keys above this are masked for every row of the wave
  int wave_first_limit;    // keys up to this are visible to every row of the wave
  float sl2;
};

// P^T operands (bf16) of one 32-key half; returns this lane's share of the
// half's row sum, taken from the rounded probabilities that the P.V product
// uses (pairs summed by v_dot2c_f32_bf16 against (1, 1)).
template <int D>
__device__ __forceinline__ float softmax_half(const WaveState<D> &w, const f32x16 &sacc, float m_use,
                                              bf16x8 (&pf)[2]) {
#pragma unroll
  for (int r = 0; r < 16; ++r) pf[r >> 3][r & 7] = (__bf16)fast_exp2(__builtin_fmaf(sacc[r], w.sl2, -m_use));
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float ps[2] = {0.f, 0.f};
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const bf16x2 pr = {pf[j >> 2][2 * (j & 3)], pf[j >> 2][2 * (j & 3) + 1]};
    ps[j & 1] = __builtin_amdgcn_fdot2_f32_bf16(pr, ones, ps[j & 1], false);
  }
  return ps[0] + ps[1];
}

// O^T += V^T P^T over the 2 x 16 keys of one half tile.
template <int D>
__device__ __forceinline__ void pv_half(WaveState<D> &w, const unsigned char *vs, const bf16x8 (&pf)[2]) {
  constexpr int ROWB = Geo<D>::ROWB, DB = Geo<D>::DB;
  // all transposed V reads of the half tile before its MFMAs
  bf16x8 a[2][DB];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int db = 0; db < DB; ++db) a[c][db] = tr_pair(vs + c * 16 * ROWB, w.voff[db][0], w.voff[db][1]);
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int db = 0; db < DB; ++db) w.oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[c][db], pf[c], w.oacc[db], 0, 0, 0);
}

// Raise the running max if this half's max grew by more than the slack
// (wave-uniform decision), rescaling O and the row sum.
template <int D>
__device__ __forceinline__ void raise_to(WaveState<D> &w, float mt) {
  const float m_new = fmaxf(w.m_run, mt);
  const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(w.m_run - m_new);
  w.m_run = m_new;
  w.l_run *= alpha;
#pragma unroll
  for (int db = 0; db < Geo<D>::DB; ++db) w.oacc[db] *= alpha;
}
template <int D>
__device__ __forceinline__ void maybe_raise(WaveState<D> &w, float mt) {
  if (__builtin_amdgcn_ballot_w64(mt > w.m_run + kRescaleSlack) != 0) raise_to<D>(w, mt);
}
template <int D>
__device__ __forceinline__ float half_max(const WaveState<D> &w, const f32x16 &sacc) {
  float mx = sacc[0];
#pragma unroll
  for (int r = 1; r < 16; ++r) mx = fmaxf(mx, sacc[r]);
  return pair_max(mx) * w.sl2;
}

// One 64-key tile: S^T = K Q^T, online softmax, O^T update. MASK selects the
// diagonal-tile variant (causal mask, possibly a fully masked second half).
// Full tiles keep one running max per 32-key half, so the S MFMAs of half 1
// overlap the softmax of half 0 and the P.V MFMAs of half 0 overlap the max of
// half 1.
template <int D, bool MASK>
__device__ __forceinline__ void tile_math(WaveState<D> &w, const unsigned char *ks, const unsigned char *vs, int kb) {
  constexpr int ROWB = Geo<D>::ROWB, DS = Geo<D>::DS;
  if (!MASK) {
    bf16x8 kf[2][DS];
#pragma unroll
    for (int b2 = 0; b2 < 2; ++b2)
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) kf[b2][ds] = *reinterpret_cast<const bf16x8 *>(ks + b2 * 32 * ROWB + w.koff[ds]);
    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0][ds], w.qf[ds], s0, 0, 0, 0);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[1][ds], w.qf[ds], s1, 0, 0, 0);
    bf16x8 pf0[2];
    float ps0 = softmax_half<D>(w, s0, w.m_run, pf0);
    // scheduling: K reads of half 0, the S MFMAs of half 0 each beside a K
    // read of half 1, then the S MFMAs of half 1 each beside a sixth of the
    // softmax of half 0
    __builtin_amdgcn_sched_group_barrier(0x100, DS, 0);
#pragma unroll
    for (int i = 0; i < DS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#pragma unroll
    for (int i = 0; i < DS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
    }
    if (__builtin_amdgcn_ballot_w64(!(ps0 <= kHalfSumLimit)) != 0) {
      raise_to<D>(w, half_max<D>(w, s0));
      ps0 = softmax_half<D>(w, s0, w.m_run, pf0);
    }
    w.l_run += ps0;
    pv_half<D>(w, vs, pf0);
    bf16x8 pf1[2];
    float ps1 = softmax_half<D>(w, s1, w.m_run, pf1);
    if (__builtin_amdgcn_ballot_w64(!(ps1 <= kHalfSumLimit)) != 0) {
      raise_to<D>(w, half_max<D>(w, s1));
      ps1 = softmax_half<D>(w, s1, w.m_run, pf1);
    }
    w.l_run += ps1;
    pv_half<D>(w, vs + 32 * ROWB, pf1);
    return;
  }
  const bool second = kb + 32 <= w.wave_last_key;
  f32x16 sacc[2];
#pragma unroll
  for (int b2 = 0; b2 < 2; ++b2) {
    if (b2 == 1 && !second) {
      sacc[1] = f32x16{};
      continue;
    }
    bf16x8 kf[DS];
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) kf[ds] = *reinterpret_cast<const bf16x8 *>(ks + b2 * 32 * ROWB + w.koff[ds]);
    sacc[b2] = f32x16{};
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) sacc[b2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ds], w.qf[ds], sacc[b2], 0, 0, 0);
  }
#pragma unroll
  for (int b2 = 0; b2 < 2; ++b2) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = kb + 32 * b2 + 8 * (r >> 2) + 4 * w.half + (r & 3);
      if (key > w.limit) sacc[b2][r] = -INFINITY;
    }
  }
  float mx = fmaxf(sacc[0][0], sacc[1][0]);
#pragma unroll
  for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(sacc[0][r], sacc[1][r]));
  maybe_raise<D>(w, pair_max(mx) * w.sl2);
  const float m_use = (w.m_run == -INFINITY) ? 0.f : w.m_run;
  bf16x8 pf0[2], pf1[2];
  w.l_run += softmax_half<D>(w, sacc[0], m_use, pf0);
  pv_half<D>(w, vs, pf0);
  if (second) {
    w.l_run += softmax_half<D>(w, sacc[1], m_use, pf1);
    pv_half<D>(w, vs + 32 * ROWB, pf1);
  }
}

// One 64-key tile read from buffer `ks`/`vs`; the DMA of the next tile goes to
// `nk`/`nv`. The buffers are distinct LDS objects at each call site.
template <int D>
__device__ __forceinline__ void tile_step(WaveState<D> &w, const unsigned char *ks, const unsigned char *vs,
                                          unsigned char *nk, unsigned char *nv, int kb, bool prefetch) {
  // Wait for this wave's DMA of this tile (the only vector-memory work in
  // flight; the compiler does not count LDS DMA as a store to release), then
  // barrier: every wave's DMA has landed and every wave is done reading the
  // other buffer (previous tile). The fences of __syncthreads keep the
  // compiler from moving LDS reads or the next DMA across the barrier.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt and lgkmcnt left at their maxima
  __syncthreads();
  if (prefetch) dma_tile<Geo<D>::IPW>(w.kg, w.vg, kb + kBN, w.n_keys, w.kv_row_bytes, nk, nv, w.wave, w.dma_k, w.dma_v);
  if (kb > w.wave_last_key) return;               // the whole tile is masked for this wave
  if (kb + kBN - 1 > w.wave_first_limit) tile_math<D, true>(w, ks, vs, kb);
  else tile_math<D, false>(w, ks, vs, kb);
}

// One job: the work of launch slot `slot` of XCD `xcd` (one query head of one
// work group, or one packed stage-2 unit group), run by the whole workgroup.
template <int D, int KIND>
__device__ __forceinline__ void attn_job(const AttnLaunch &p, const int xcd, const int slot, unsigned char *k_lds0,
                                         unsigned char *v_lds0, unsigned char *k_lds1, unsigned char *v_lds1) {
  using Gm = Geo<D>;
  constexpr int ROWB = Gm::ROWB, CH = Gm::CH, TILE = Gm::TILE, IPW = Gm::IPW, DS = Gm::DS, DB = Gm::DB;
  constexpr int RPI = Gm::RPI;
  // ---- which work -----------------------------------------------------------
  // A work group is the G heads that share one KV head, for one entry, query
  // block and key split. When Hkv divides the 8 XCDs, each XCD serves one KV
  // head (8/Hkv XCDs per head, dealt alternately a, b, b, a, ...), so every L2
  // holds the K/V of a single head;
  // otherwise work groups are dealt to the XCDs round-robin. Within an XCD,
  // work groups run heaviest first, and the G heads of a work group are
  // consecutive workgroups of that XCD.
  const int G = p.group, WPG = p.wgs_per_group;
  const int hl = slot % WPG;
  int g, lam;  // KV head, index of the work group among that head's work groups
  if (kXcds % p.hkv == 0) {
    const int xph = kXcds / p.hkv;
    g = xcd / xph;
    // work groups of a head are dealt to its xph XCDs in boustrophedon order
    // (a, b, b, a, ...), so the XCDs get equal shares of the heaviest-first list
    const int q = slot / WPG, r = xcd % xph;
    lam = q * xph + ((q & 1) ? xph - 1 - r : r);
    if (lam * p.hkv >= p.n_groups) return;
  } else {
    const int gamma = (slot / WPG) * kXcds + xcd;
    if (gamma >= p.n_groups) return;
    g = gamma % p.hkv;
    lam = gamma / p.hkv;
  }
  int ei = 0;
  while (ei + 1 < p.n_entries && p.e[ei + 1].group0 <= lam * p.hkv) ++ei;
  const AttnEntry &E = p.e[ei];
  const int ll = lam - E.group0 / p.hkv;
  const int s = ll % E.n_splits;
  const int mb = E.mb_hi - ll / E.n_splits;

  const int n_rows = E.n_rows;
  const int n_keys = E.n_keys;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  // this wave's query head and first row, and the workgroup's last row
  int h, wrow0, row_last;
  if (KIND == 1 && WPG == 1) {
    // packed units (the split-key kernel always runs packed; with G = 1 the
    // units of a workgroup are 4 consecutive row blocks of one head): unit u = (head hl_u, 32-row block rb_u), u = hl_u * n_rb + rb_u
    const int n_rb = (n_rows + 31) / 32, n_units = G * n_rb;
    const int u = mb * 4 + wave;
    h = g * G + min(u, n_units - 1) / n_rb;
    wrow0 = u < n_units ? (u % n_rb) * 32 : n_rows;  // a wave past the last unit has no rows
    row_last = 0;
    for (int j = 0; j < 4; ++j) {
      const int uj = mb * 4 + j;
      if (uj < n_units) row_last = max(row_last, min((uj % n_rb) * 32 + 31, n_rows - 1));
    }
  } else {
    h = g * G + hl;
    wrow0 = mb * kAttnBM + wave * 32;
    row_last = min(mb * kAttnBM + kAttnBM, n_rows) - 1;
  }
  const int k_begin = s * E.split_keys;
  const int k_end = min(min(k_begin + E.split_keys, n_keys), row_limit(E, row_last) + 1);
  const int n_tiles = k_end > k_begin ? (k_end - k_begin + kBN - 1) / kBN : 0;

  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int my_row = wrow0 + l32;
  // keys above this are masked for the whole wave (a wave past the last row has none)
  const int wave_last_key = wrow0 < n_rows ? row_limit(E, wrow0 + 31) : -1;

  WaveState<D> w;
  w.kg = static_cast<const unsigned char *>(E.k);
  w.vg = static_cast<const unsigned char *>(E.v);
  w.n_keys = n_keys;
  w.kv_row_bytes = p.hkv * D * 2;
  w.limit = row_limit(E, my_row);
  w.wave_last_key = wave_last_key;
  w.wave_first_limit = row_limit(E, wrow0);
  w.half = half;
  w.wave = wave;
  w.sl2 = p.scale_log2;
  w.m_run = -INFINITY;
  w.l_run = 0.f;
#pragma unroll
  for (int db = 0; db < DB; ++db) w.oacc[db] = f32x16{};
  {
    const __bf16 *qp = static_cast<const __bf16 *>(E.q) + ((size_t)my_row * p.hq + h) * D + 8 * half;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      w.qf[ds] = my_row < n_rows ? *reinterpret_cast<const bf16x8 *>(qp + 16 * ds) : bf16x8{};
  }
#pragma unroll
  for (int i = 0; i < IPW; ++i) {
    const int r = (wave * IPW + i) * RPI + lane / CH;
    const int pc = lane % CH;
    w.dma_k[i] = r * w.kv_row_bytes + g * D * 2 + ((pc ^ swz_k(r, CH)) << 4);
    w.dma_v[i] = r * w.kv_row_bytes + g * D * 2 + ((pc ^ swz_v(r, CH)) << 4);
  }
#pragma unroll
  for (int ds = 0; ds < DS; ++ds) w.koff[ds] = l32 * ROWB + (((2 * ds + half) ^ swz_k(l32, CH)) << 4);
  {
    const int grp = lane >> 4, j = lane & 15;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int key = 8 * b + 4 * (grp >> 1) + (j >> 2);
      const int sw = swz_v(key, CH);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const int lc = 4 * db + 2 * (grp & 1) + ((j & 3) >> 1);
        w.voff[db][b] = key * ROWB + ((lc ^ sw) << 4) + 8 * (j & 1);
      }
    }
  }

  if (n_tiles > 0) dma_tile<IPW>(w.kg, w.vg, k_begin, n_keys, w.kv_row_bytes, k_lds0, v_lds0, wave, w.dma_k, w.dma_v);
  for (int t = 0; t < n_tiles; t += 2) {
    // even tiles live in buffer 0, odd tiles in buffer 1
    int kb = k_begin + t * kBN;
    tile_step<D>(w, k_lds0, v_lds0, k_lds1, v_lds1, kb, t + 1 < n_tiles);
    if (t + 1 < n_tiles) {
      kb += kBN;
      tile_step<D>(w, k_lds1, v_lds1, k_lds0, v_lds0, kb, t + 2 < n_tiles);
    }
  }

  // ---- epilogue ---------------------------------------------------------------
  const float l_tot = pair_sum(w.l_run);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_nat = l_tot > 0.f ? (w.m_run + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
  // Rows go out through LDS so that every store is a 16-byte piece of a
  // contiguous row (a lane holds 4-feature pieces of one row, spread over the
  // row). Each wave stages in its own quarter of the stage buffer that did
  // not hold the last tile: every wave finished reading it before the last
  // barrier and no copy targets it any more.
  unsigned char *stg = ((n_tiles & 1) ? (wave < 2 ? k_lds1 : v_lds1) : (wave < 2 ? k_lds0 : v_lds0)) +
                       (wave & 1) * (TILE / 2);
  const int wrow = wrow0;  // first row of this wave
  if (E.n_splits == 1 && E.o != nullptr) {
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 v;
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = (__bf16)(w.oacc[db][4 * q4 + t] * inv);
        stage_put<D>(stg, l32, 4 * db + q4, 8 * half, v);
      }
    store_rows<D>(stg, lane, wrow, n_rows, [&](int r) {
      return static_cast<unsigned char *>(E.o) + ((size_t)r * p.hq + h) * D * 2;
    });
    if (E.o2 != nullptr)
      store_rows<D>(stg, lane, wrow, n_rows, [&](int r) {
        const int64_t r2 = E.o2_row0 + (E.o2_idx ? E.o2_idx[r] : r);
        return static_cast<unsigned char *>(E.o2) + ((size_t)r2 * p.hq + h) * D * 2;
      });
    if (E.lse != nullptr && half == 0 && my_row < n_rows) E.lse[(size_t)h * E.lse_stride + my_row] = lse_nat;
  } else {
    // bf16 partials (the normalised split output, like a final output row)
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        bf16x4 v;
#pragma unroll
        for (int t = 0; t < 4; ++t) v[t] = (__bf16)(w.oacc[db][4 * q4 + t] * inv);
        stage_put<D>(stg, l32, 4 * db + q4, 8 * half, v);
      }
    store_rows<D>(stg, lane, wrow, n_rows, [&](int r) {
      const size_t prow = (size_t)r * E.n_splits + s;
      return static_cast<unsigned char *>(E.part_o) + (prow * p.hq + h) * D * 2;
    });
    if (half == 0 && my_row < n_rows) E.part_lse[((size_t)my_row * E.n_splits + s) * p.hq + h] = lse_nat;
  }
}

// Launch shape: the first pair_wgs workgroups of each XCD each run two jobs,
// slot u and slot 2*pair_wgs-1-u of the XCD's heaviest-first list (a heavy job
// with a light one, so that their sums are nearly equal), and every further
// workgroup runs one of the remaining, lightest slots. With pair_wgs = 0 each
// workgroup runs one slot.
template <int D, int KIND>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_bf16_kernel(const AttnLaunch p) {
  constexpr int TILE = Geo<D>::TILE;
  // separate objects per stage and tensor: lets the compiler see that the DMA
  // into one buffer does not alias reads of another
  __shared__ __attribute__((aligned(1024))) unsigned char k_lds0[TILE];
  __shared__ __attribute__((aligned(1024))) unsigned char v_lds0[TILE];
  __shared__ __attribute__((aligned(1024))) unsigned char k_lds1[TILE];
  __shared__ __attribute__((aligned(1024))) unsigned char v_lds1[TILE];
  const int xcd = blockIdx.x % kXcds;
  const int u = blockIdx.x / kXcds;
  const bool paired = u < p.pair_wgs;
  const int first = paired ? u : u + p.pair_wgs;
  const int second = 2 * p.pair_wgs - 1 - u;
  const int n_jobs = (paired && second < p.slots_per_xcd) ? 2 : 1;
  for (int j = 0; j < n_jobs; ++j) {
    if (j) __syncthreads();  // every wave is done with the LDS buffers of the first job
    attn_job<D, KIND>(p, xcd, j ? second : first, k_lds0, v_lds0, k_lds1, v_lds1);
  }
}

template <int D>
hipError_t launch_t(AttnKind kind, const AttnLaunch &p0, hipStream_t st) {
  AttnLaunch p = p0;
  // slots per XCD: work groups per XCD times the G heads of a work group
  int per_xcd;
  if (kXcds % p.hkv == 0) {
    const int xph = kXcds / p.hkv, per_head = p.n_groups / p.hkv;
    per_xcd = (per_head + xph - 1) / xph;
  } else {
    per_xcd = (p.n_groups + kXcds - 1) / kXcds;
  }
  const int slots = p.wgs_per_group * per_xcd;
  // Causal self attention: the heaviest 2 * kResidentPerXcd slots of an XCD
  // run in heavy/light pairs (see the kernel). Slots are in heaviest-first
  // order within an entry, and entries heaviest request first, so the pairing
  // is used when the first entry alone fills those slots.
  const int xph = kXcds % p.hkv == 0 ? kXcds / p.hkv : 0;
  const int first_groups = xph ? p.e[0].mb_count / xph : p.e[0].mb_count * p.hkv / kXcds;
  p.slots_per_xcd = slots;
  p.pair_wgs = (kind == AttnKind::kSelf && p.e[0].n_splits == 1 &&
                first_groups * p.wgs_per_group >= 2 * kResidentPerXcd)
                   ? kResidentPerXcd
                   : 0;
  const int wgs = p.pair_wgs ? p.pair_wgs + std::max(0, slots - 2 * p.pair_wgs) : slots;
  const dim3 grid(kXcds * wgs), block(kAttnThreads);
  switch (kind) {
    case AttnKind::kSelf: attn_bf16_kernel<D, 0><<<grid, block, 0, st>>>(p); break;
    default: attn_bf16_kernel<D, 1><<<grid, block, 0, st>>>(p); break;
  }
  return hipGetLastError();
}

// ---- merge of the stage-2 split partials ---------------------------------------
//
// Merge of the bf16 split partials: one wave per (question row, query head).
// Lane = split group * CHN + chunk: each lane accumulates one 8-feature chunk
// over every SG-th split (online log-sum-exp), then the split groups combine
// across lanes.
template <int D>
__global__ __launch_bounds__(256) void qdoc_merge_kernel(const MergeLaunch p) {
  constexpr int CHN = D / 8, SG = 64 / CHN;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, c = lane % CHN, sg = lane / CHN;
  const int row = item / p.hq, h = item % p.hq;
  if (row >= p.total_rows) return;  // whole waves leave together
  int ei = 0;
  while (ei + 1 < p.n_entries && p.e[ei + 1].row0 <= row) ++ei;
  const MergeEntry &E = p.e[ei];
  const int r = row - E.row0;
  const int S = E.n_splits;
  const size_t prow0 = (size_t)r * S;
  const float *lse = E.part_lse + prow0 * p.hq + h;
  const __bf16 *src = static_cast<const __bf16 *>(E.part_o) + (prow0 * p.hq + h) * D + 8 * c;
  const size_t sstride = (size_t)p.hq * D;
  constexpr int U = 8;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, wsum = 0.f;
  for (int s0 = sg; s0 < S; s0 += SG * U) {
    float ls[U];
    bf16x8 po[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int sx = s0 + u * SG;
      if (sx < S) {
        ls[u] = lse[(size_t)sx * p.hq];
        po[u] = *reinterpret_cast<const bf16x8 *>(src + sx * sstride);
      } else {
        ls[u] = -INFINITY;
        po[u] = bf16x8{};
      }
    }
    float mc = m;
#pragma unroll
    for (int u = 0; u < U; ++u) mc = fmaxf(mc, ls[u]);
    const float a = (m == -INFINITY) ? 0.f : __expf(m - mc);
    wsum *= a;
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] *= a;
    m = mc;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float wt = (ls[u] == -INFINITY) ? 0.f : __expf(ls[u] - m);
      wsum += wt;
#pragma unroll
      for (int k = 0; k < 8; ++k) acc[k] += wt * (float)po[u][k];
    }
  }
  // combine the SG split groups (lanes c, c + CHN, c + 2 CHN, ...)
#pragma unroll
  for (int off = CHN; off < 64; off *= 2) {
    const float m2 = __shfl_xor(m, off, 64), w2 = __shfl_xor(wsum, off, 64);
    const float mm = fmaxf(m, m2);
    const float a = (m == -INFINITY) ? 0.f : __expf(m - mm);
    const float b = (m2 == -INFINITY) ? 0.f : __expf(m2 - mm);
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = acc[k] * a + __shfl_xor(acc[k], off, 64) * b;
    wsum = wsum * a + w2 * b;
    m = mm;
  }
  if (sg != 0) return;
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  bf16x8 out;
#pragma unroll
  for (int k = 0; k < 8; ++k) out[k] = (__bf16)(acc[k] * inv);
  *reinterpret_cast<bf16x8 *>(static_cast<__bf16 *>(E.o) + ((size_t)r * p.hq + h) * D + 8 * c) = out;
  if (E.o2 != nullptr)
    *reinterpret_cast<bf16x8 *>(static_cast<__bf16 *>(E.o2) + ((size_t)(E.o2_row0 + r) * p.hq + h) * D + 8 * c) = out;
  if (E.lse != nullptr && c == 0) E.lse[(size_t)h * E.lse_stride + r] = wsum > 0.f ? m + __logf(wsum) : -INFINITY;
}

template <int D>
hipError_t launch_qdoc_merge_t(const MergeLaunch &p, hipStream_t st) {
  const int64_t items = (int64_t)p.total_rows * p.hq;
  qdoc_merge_kernel<D><<<dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st>>>(p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_bf16(int head_dim, AttnKind kind, const AttnLaunch &p, hipStream_t st) {
  if (p.n_groups <= 0) return hipSuccess;
  return head_dim == 128 ? launch_t<128>(kind, p, st) : launch_t<64>(kind, p, st);
}

hipError_t launch_qdoc_merge_bf16(int head_dim, const MergeLaunch &p, hipStream_t st) {
  if (p.total_rows <= 0) return hipSuccess;
  return head_dim == 128 ? launch_qdoc_merge_t<128>(p, st) : launch_qdoc_merge_t<64>(p, st);
}

}  // namespace daf
