// Causal GQA flash attention for both DAF attention stages, gfx950.
//
// Stage 1 (important-token self-attention, Sec. 2 item 1) and stage 2
// (question-document attention over the hybrid cache, Sec. 2 item 2) are the
// same operation: query row i of a request sees keys 0 .. i + (n_keys -
// n_rows). Stage 1 has n_keys == n_rows (plain causal over the condensed
// sequence); stage 2 has n_rows = L_q question rows over n_keys = L_d + L_q
// cache rows. A launch carries a table of entries (requests, possibly ragged,
// each a range of query blocks with its own key split).
//
// Work decomposition. A workgroup (4 waves) owns 128 query rows of one query
// head and one key split. The G = Hq/Hkv workgroups that read the same K/V
// rows (same entry, query block, split, KV head) form a work group; work
// groups are dealt to the 8 XCDs round-robin in order (heaviest query blocks
// first), and the G members of a work group land on the same XCD so the K/V
// tile they share is fetched into that XCD's L2 once.
//
// Per workgroup. Each wave keeps its 32 query rows in registers as the B
// operand of S^T = K Q^T (v_mfma_f32_32x32x16_bf16, keys on M, query rows on
// N), so every lane owns one query row: the row max needs one exchange with
// the partner lane (lane ^ 32) and the output rescale is lane-local. The
// output is accumulated transposed, O^T += V^T P^T, with P^T taken straight
// from the S^T accumulator registers; V is staged in LDS transposed (feature
// major) with the key order permuted to match the accumulator layout, so
// every MFMA operand is one 16-byte LDS read. Softmax runs in fp32 in base 2
// with the scale folded into log2(e); probabilities are rounded to bf16 for
// the value product. The K/V tile for the next step is loaded into registers
// while the current one is consumed from LDS.
#include <math.h>

#include "daf_internal.h"

namespace daf {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Vec;
template <> struct Vec<__bf16> {
  using v8 = bf16x8;  // one MFMA operand per lane: 8 elements, 16 bytes
  using v4 = bf16x4;
};
template <> struct Vec<float> {
  using v8 = f32x8;   // 8 elements, 32 bytes
  using v4 = f32x4;
  static constexpr int kKeyTile = 32;
};

// acc += A(32x16) * B(16x32) with A, B in the 32x32x16 operand layout: lane l
// holds row/column l % 32 and k = 8 * (l / 32) + [0, 8).
__device__ __forceinline__ f32x16 mma_k16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
// fp32 inputs: eight 32x32x2 steps; step t takes element t of each lane's 8,
// so the 16-wide contraction is covered in a permuted (still complete) order.
__device__ __forceinline__ f32x16 mma_k16(f32x8 a, f32x8 b, f32x16 c) {
#pragma unroll
  for (int t = 0; t < 8; ++t)
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[t], b[t], c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Position of key `key` (0 .. tile-1) in a row of the transposed V tile.
// Within each 16-key group the accumulator of S^T hands lane half 0 the keys
// {0-3, 8-11} and half 1 the keys {4-7, 12-15}; storing the quads in the order
// 0, 2, 1, 3 makes each half's 8 keys contiguous.
__device__ __forceinline__ int vt_pos(int key) {
  const int quad = (key >> 2) & 3;
  const int qp = (quad == 1) ? 2 : (quad == 2) ? 1 : quad;
  return (key & ~15) + (qp << 2) + (key & 3);
}

template <typename T, int D, int KIND>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_fwd_kernel(const AttnLaunch p) {
  using V8 = typename Vec<T>::v8;
  using V4 = typename Vec<T>::v4;
  constexpr int BN = Vec<T>::kKeyTile;   // keys per step
  constexpr int PAD = 16 / sizeof(T);    // 16 bytes of padding per LDS row
  constexpr int KLD = D + PAD;           // K tile row pitch (elements)
  constexpr int VLD = BN + PAD;          // V^T tile row pitch (elements)
  constexpr int DS = D / 16;             // contraction steps of S^T
  constexpr int DB = D / 32;             // 32-feature output blocks
  constexpr int NKB = BN / 32;           // 32-key blocks per step
  constexpr int KU = BN * D / 8;         // 8-element K units per tile
  constexpr int KUT = (KU + kAttnThreads - 1) / kAttnThreads;
  constexpr int VU = (BN / 4) * (D / 8); // (4 keys x 8 features) V units per tile
  constexpr int VUT = (VU + kAttnThreads - 1) / kAttnThreads;

  __shared__ __attribute__((aligned(16))) T Ks[BN * KLD];
  __shared__ __attribute__((aligned(16))) T Vt[D * VLD];

  // ---- which work: XCD-aware deal of work groups ----------------------------
  const int G = p.group;
  const int xcd = blockIdx.x % kXcds;
  const int slot = blockIdx.x / kXcds;
  const int gamma = (slot / G) * kXcds + xcd;
  const int hl = slot % G;
  if (gamma >= p.n_groups) return;
  int ei = 0;
  while (ei + 1 < p.n_entries && p.e[ei + 1].group0 <= gamma) ++ei;
  const AttnEntry &E = p.e[ei];
  int gl = gamma - E.group0;
  const int g = gl % p.hkv;
  gl /= p.hkv;
  const int s = gl % E.n_splits;
  gl /= E.n_splits;
  const int mb = E.mb_hi - gl;
  const int h = g * G + hl;

  const int n_rows = E.n_rows;
  const int row0 = mb * kAttnBM;
  const int row_last = min(row0 + kAttnBM, n_rows) - 1;
  const int k_begin = s * E.split_keys;
  const int k_end = min(min(k_begin + E.split_keys, E.n_keys), row_limit(E, row_last) + 1);

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int l32 = lane & 31;
  const int half = lane >> 5;
  const int wrow0 = row0 + wave * 32;
  const int my_row = wrow0 + l32;

  // ---- Q fragments (B operand of S^T): row my_row, features 16*ds + 8*half --
  V8 qf[DS];
  {
    const T *qp = static_cast<const T *>(E.q) + ((size_t)my_row * p.hq + h) * D + 8 * half;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      if (my_row < n_rows) qf[ds] = *reinterpret_cast<const V8 *>(qp + 16 * ds);
      else qf[ds] = V8{};
    }
  }

  const T *kg = static_cast<const T *>(E.k);
  const T *vg = static_cast<const T *>(E.v);
  const size_t kv_row = (size_t)p.hkv * D;  // elements between consecutive keys
  const int n_keys = E.n_keys;

  V8 kreg[KUT];
  V8 vreg[VUT][4];
  auto load_tile = [&](int kb) {
#pragma unroll
    for (int i = 0; i < KUT; ++i) {
      const int u = tid + i * kAttnThreads;
      if (KU % kAttnThreads == 0 || u < KU) {
        const int key = u / (D / 8), dc = u % (D / 8);
        const int kk = kb + key;
        kreg[i] = kk < n_keys ? *reinterpret_cast<const V8 *>(kg + kk * kv_row + (size_t)g * D + dc * 8)
                              : V8{};
      }
    }
#pragma unroll
    for (int i = 0; i < VUT; ++i) {
      const int u = tid + i * kAttnThreads;
      if (VU % kAttnThreads == 0 || u < VU) {
        const int kq = u % (BN / 4), dc = u / (BN / 4);
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int kk = kb + 4 * kq + t;
          vreg[i][t] = kk < n_keys ? *reinterpret_cast<const V8 *>(vg + kk * kv_row + (size_t)g * D + dc * 8)
                                   : V8{};
        }
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KUT; ++i) {
      const int u = tid + i * kAttnThreads;
      if (KU % kAttnThreads == 0 || u < KU) {
        const int key = u / (D / 8), dc = u % (D / 8);
        *reinterpret_cast<V8 *>(&Ks[key * KLD + dc * 8]) = kreg[i];
      }
    }
#pragma unroll
    for (int i = 0; i < VUT; ++i) {
      const int u = tid + i * kAttnThreads;
      if (VU % kAttnThreads == 0 || u < VU) {
        const int kq = u % (BN / 4), dc = u / (BN / 4);
        const int pos = vt_pos(4 * kq);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          V4 w;
          w[0] = vreg[i][0][e];
          w[1] = vreg[i][1][e];
          w[2] = vreg[i][2][e];
          w[3] = vreg[i][3][e];
          *reinterpret_cast<V4 *>(&Vt[(dc * 8 + e) * VLD + pos]) = w;
        }
      }
    }
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY;  // running row max (scaled, base 2); equal in both halves
  float l_run = 0.f;        // this lane's share of the row sum

  const float sl2 = p.scale_log2;
  const int limit = row_limit(E, my_row);  // last visible key of this lane's row
  const int wave_first_limit = row_limit(E, wrow0);  // keys up to this are visible to every row

  if (k_begin < k_end) load_tile(k_begin);
  for (int kb = k_begin; kb < k_end; kb += BN) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (kb + BN < k_end) load_tile(kb + BN);

    // S^T = K Q^T, 32 keys x 32 rows per block
    f32x16 sacc[NKB];
#pragma unroll
    for (int b2 = 0; b2 < NKB; ++b2) {
      sacc[b2] = f32x16{};
      const T *kr = &Ks[(b2 * 32 + l32) * KLD + 8 * half];
#pragma unroll
      for (int ds = 0; ds < DS; ++ds)
        sacc[b2] = mma_k16(*reinterpret_cast<const V8 *>(kr + 16 * ds), qf[ds], sacc[b2]);
    }

    // scale, causal mask, row max
    const bool need_mask = (kb + BN - 1) > wave_first_limit;
    float mloc = -INFINITY;
#pragma unroll
    for (int b2 = 0; b2 < NKB; ++b2) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x = sacc[b2][r] * sl2;
        if (need_mask) {
          const int key = kb + b2 * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key > limit) x = -INFINITY;
        }
        sacc[b2][r] = x;
        mloc = fmaxf(mloc, x);
      }
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float alpha = fast_exp2(m_run - m_use);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int b2 = 0; b2 < NKB; ++b2) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float e = fast_exp2(sacc[b2][r] - m_use);
        sacc[b2][r] = e;
        psum += e;
      }
    }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] *= alpha;

    // P^T operands: 16 keys each, straight from the accumulator registers
    V8 pf[BN / 16];
#pragma unroll
    for (int c = 0; c < BN / 16; ++c) {
#pragma unroll
      for (int t = 0; t < 8; ++t) pf[c][t] = (T)sacc[c >> 1][(c & 1) * 8 + t];
    }
    // O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const T *vr = &Vt[(db * 32 + l32) * VLD + 8 * half];
#pragma unroll
      for (int c = 0; c < BN / 16; ++c)
        oacc[db] = mma_k16(*reinterpret_cast<const V8 *>(vr + 16 * c), pf[c], oacc[db]);
    }
  }

  // ---- epilogue ---------------------------------------------------------------
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
  const float lse_nat = l_tot > 0.f ? (m_run + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
  if (my_row >= n_rows) return;
  if (E.n_splits == 1 && E.o != nullptr) {
    T *op = static_cast<T *>(E.o) + ((size_t)my_row * p.hq + h) * D + 4 * half;
    T *op2 = nullptr;
    if (E.o2 != nullptr) {
      const int64_t r2 = E.o2_row0 + (E.o2_idx ? E.o2_idx[my_row] : my_row);
      op2 = static_cast<T *>(E.o2) + ((size_t)r2 * p.hq + h) * D + 4 * half;
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        V4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = (T)(oacc[db][4 * q4 + t] * inv);
        *reinterpret_cast<V4 *>(op + db * 32 + 8 * q4) = w;
        if (op2) *reinterpret_cast<V4 *>(op2 + db * 32 + 8 * q4) = w;
      }
    }
    if (E.lse != nullptr && half == 0) E.lse[(size_t)h * E.lse_stride + my_row] = lse_nat;
  } else {
    const size_t prow = (size_t)my_row * E.n_splits + s;
    float *op = static_cast<float *>(E.part_o) + (prow * p.hq + h) * D + 4 * half;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        f32x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = oacc[db][4 * q4 + t] * inv;
        *reinterpret_cast<f32x4 *>(op + db * 32 + 8 * q4) = w;
      }
    }
    if (half == 0) E.part_lse[prow * p.hq + h] = lse_nat;
  }
}

// Log-sum-exp merge of the key splits. Each (query row, head) item gets two
// groups of D/4 threads, each thread owning 4 features; group j merges its
// half of the splits (m = max_s lse_s, w_s = exp(lse_s - m), acc = sum_s w_s
// O_s, wsum = sum_s w_s), then the two halves are combined across the lanes
// (lane ^ D/4) and the first group writes O = acc / wsum and lse = m + log
// wsum. Split partials are read with 16-byte loads, all of a half's splits in
// flight at once for up to 32 splits (one round trip to memory).
template <typename T, int D>
__global__ __launch_bounds__(256) void lse_merge_kernel(const MergeLaunch p) {
  constexpr int TPI = D / 4;              // threads per item and split half
  constexpr int IPB = 256 / (2 * TPI);    // items per block
  const int item = blockIdx.x * IPB + threadIdx.x / (2 * TPI);
  const int hs = (threadIdx.x / TPI) & 1;  // which half of the splits
  const int t = threadIdx.x % TPI;
  const int row = item / p.hq, h = item % p.hq;
  if (row >= p.total_rows) return;  // both halves of an item leave together
  int ei = 0;
  while (ei + 1 < p.n_entries && p.e[ei + 1].row0 <= row) ++ei;
  const MergeEntry &E = p.e[ei];
  const int r = row - E.row0;
  const int S = E.n_splits;
  const int per_half = (S + 1) / 2;
  const int sb = hs * per_half, se = min(S, sb + per_half);
  const size_t prow0 = (size_t)r * S;
  const float *lse = E.part_lse + prow0 * p.hq + h;
  // partial outputs in the output dtype T: 4 features (8 or 16 bytes) per thread and split
  const T *src = static_cast<const T *>(E.part_o) + (prow0 * p.hq + h) * D + 4 * t;
  const size_t split_stride = (size_t)p.hq * D;
  constexpr int U = 16;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY, wsum = 0.f;
  for (int s0 = sb; s0 < se; s0 += U) {
    float ls[U];
    f32x4 po[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < se) {
        ls[u] = lse[(size_t)(s0 + u) * p.hq];
        const typename Vec<T>::v4 v = *reinterpret_cast<const typename Vec<T>::v4 *>(src + (s0 + u) * split_stride);
#pragma unroll
        for (int j = 0; j < 4; ++j) po[u][j] = (float)v[j];
      } else {
        ls[u] = -INFINITY;
        po[u] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    float mc = m;
#pragma unroll
    for (int u = 0; u < U; ++u) mc = fmaxf(mc, ls[u]);
    // rescale what earlier chunks accumulated to the new max
    const float a = (m == -INFINITY) ? 0.f : __expf(m - mc);
    acc *= a;
    wsum *= a;
    m = mc;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float w = (ls[u] == -INFINITY) ? 0.f : __expf(ls[u] - m);
      wsum += w;
      acc += w * po[u];
    }
  }
  // combine with the other half
  {
    const float m2 = __shfl_xor(m, TPI, 64), w2 = __shfl_xor(wsum, TPI, 64);
    f32x4 acc2;
#pragma unroll
    for (int j = 0; j < 4; ++j) acc2[j] = __shfl_xor(acc[j], TPI, 64);
    const float mm = fmaxf(m, m2);
    const float a = (m == -INFINITY) ? 0.f : __expf(m - mm);
    const float b = (m2 == -INFINITY) ? 0.f : __expf(m2 - mm);
    wsum = wsum * a + w2 * b;
    acc = acc * a + acc2 * b;
    m = mm;
  }
  if (hs != 0) return;
  const float inv = 1.f / wsum;
  T *dst = static_cast<T *>(E.o) + ((size_t)r * p.hq + h) * D + 4 * t;
  typename Vec<T>::v4 o;
#pragma unroll
  for (int j = 0; j < 4; ++j) o[j] = (T)(acc[j] * inv);
  *reinterpret_cast<typename Vec<T>::v4 *>(dst) = o;
  if (E.o2 != nullptr)
    *reinterpret_cast<typename Vec<T>::v4 *>(static_cast<T *>(E.o2) +
                                             ((size_t)(E.o2_row0 + r) * p.hq + h) * D + 4 * t) = o;
  if (E.lse != nullptr && t == 0) E.lse[(size_t)h * E.lse_stride + r] = m + __logf(wsum);
}

template <typename T, int D>
hipError_t launch_attn_t(AttnKind kind, const AttnLaunch &p, hipStream_t st) {
  const int slots = p.wgs_per_group * ((p.n_groups + kXcds - 1) / kXcds);
  const dim3 grid(kXcds * slots), block(kAttnThreads);
  switch (kind) {
    case AttnKind::kSelf: attn_fwd_kernel<T, D, 0><<<grid, block, 0, st>>>(p); break;
    default: attn_fwd_kernel<T, D, 1><<<grid, block, 0, st>>>(p); break;
  }
  return hipGetLastError();
}

template <typename T, int D>
hipError_t launch_merge_t(const MergeLaunch &p, hipStream_t st) {
  const int items = p.total_rows * p.hq;
  constexpr int IPB = 256 / (2 * (D / 4));
  lse_merge_kernel<T, D><<<dim3((items + IPB - 1) / IPB), dim3(256), 0, st>>>(p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(int dtype, int head_dim, AttnKind kind, const AttnLaunch &p,
                            hipStream_t st) {
  if (p.n_groups <= 0) return hipSuccess;
  if (dtype == 0) return launch_attention_bf16(head_dim, kind, p, st);
  return head_dim == 128 ? launch_attn_t<float, 128>(kind, p, st)
                         : launch_attn_t<float, 64>(kind, p, st);
}

hipError_t launch_merge(int dtype, int head_dim, const MergeLaunch &p, hipStream_t st) {
  if (p.total_rows <= 0) return hipSuccess;
  if (dtype == 0) {
    return head_dim == 128 ? launch_merge_t<__bf16, 128>(p, st) : launch_merge_t<__bf16, 64>(p, st);
  }
  return head_dim == 128 ? launch_merge_t<float, 128>(p, st) : launch_merge_t<float, 64>(p, st);
}

}  // namespace daf
