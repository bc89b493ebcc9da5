// Internal declarations shared by the DAF HIP kernels and the host library.
// gfx950 (MI355X) only: wave64, MFMA bf16 32x32x16, 8 XCDs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace daf {

constexpr int kXcds = 8;          // MI355X: 8 XCDs, workgroups dispatched round-robin
constexpr int kAttnThreads = 256; // 4 waves, 32 query rows each
constexpr int kAttnBM = 128;      // query rows per attention workgroup
constexpr int kMaxEntries = 32;   // work-table entries per attention launch (kernel argument < 4 KiB)
constexpr int kMaxRowReqs = 32;   // requests per row-movement launch
constexpr int kTargetWorkgroups = 512;  // 256 CUs x 2 resident attention workgroups
constexpr int kResidentPerXcd = 64;     // resident attention workgroups per XCD (32 CUs x 2)

// One entry of an attention launch: one request of one stage, restricted to a
// contiguous range of 128-row query blocks. Query row i (0-based in the
// entry's request) sees keys 0 .. i + (n_keys - n_rows): causal, aligned to the
// bottom right, which covers both DAF stages (stage 1: n_keys == n_rows;
// stage 2: n_keys = L_d + L_q, n_rows = L_q). With q_pos set, row i sees keys
// 0 .. q_pos[i] (queries at given positions of the key sequence).
struct AttnEntry {
  const void *q;   // [n_rows][Hq][D], row 0 of the request
  const void *k;   // [n_keys][Hkv][D]
  const void *v;
  void *o;         // [n_rows][Hq][D] final output (direct mode), else null
  float *lse;      // [Hq][lse_stride] at this request's first column, nullable
  void *part_o;    // split mode: [n_rows * n_splits][Hq][D], normalised partial outputs in the input
                   // dtype (bf16 or fp32)
  float *part_lse; // split mode: [n_rows * n_splits][Hq]
  int32_t lse_stride;
  int32_t n_rows;
  int32_t n_keys;
  int32_t mb_hi;      // heaviest (last) query block of the range (packed: unit group)
  int32_t mb_count;   // blocks mb_hi, mb_hi-1, ..., mb_hi-mb_count+1
  int32_t n_splits;   // key splits (1 = direct mode)
  int32_t split_keys; // keys per split, a multiple of the key tile
  int32_t group0;     // first work group (G query heads sharing a KV head)
  // optional second destination of each final output row (the state fusion
  // into the hidden states): row i goes to o2 row o2_row0 + (o2_idx ? o2_idx[i] : i)
  void *o2;
  const int32_t *o2_idx;
  int64_t o2_row0;
  // optional query positions: row i sees keys 0 .. q_pos[i] (strictly
  // increasing, < n_keys) instead of 0 .. i + (n_keys - n_rows)
  const int32_t *q_pos;
};

// Last key visible to query row r of entry e; rows past the end take the last
// row's limit (their outputs are never written).
__device__ __forceinline__ int row_limit(const AttnEntry &e, int r) {
  const int rr = min(r, e.n_rows - 1);
  return e.q_pos ? e.q_pos[rr] : rr + (e.n_keys - e.n_rows);
}

struct AttnLaunch;
static_assert(sizeof(AttnEntry) * kMaxEntries + 64 < 4096, "attention launch table must fit 4 KiB of kernel arguments");
struct AttnLaunch {
  int32_t hq, hkv, group;  // group = Hq / Hkv
  // workgroups per work group: G (one query head each, 128 rows) or, for the
  // bf16 split-key kernel, 1 (packed: the workgroup's 4 waves take 4
  // consecutive (head, 32-row block) units of the KV group, so every K/V tile
  // it copies serves several heads when the question is short)
  int32_t wgs_per_group;
  int32_t n_entries;
  int32_t n_groups;        // total work groups over all entries
  float scale_log2;        // softmax scale * log2(e)
  // launch shape, set by the launcher: slots per XCD, and the number of
  // workgroups per XCD that run two slots (a heavy and a light one; 0 = none)
  int32_t slots_per_xcd;
  int32_t pair_wgs;
  AttnEntry e[kMaxEntries];
};

// Log-sum-exp merge of split partials, one request per entry.
struct MergeEntry {
  const void *part_o;  // [rows * n_splits][Hq][D] in the input dtype
  const float *part_lse;
  void *o;        // [n_rows][Hq][D]
  float *lse;     // nullable, [Hq][lse_stride] at the request's first column
  int32_t lse_stride;
  int32_t n_rows;
  int32_t n_splits;
  int32_t row0;   // first global (row, head) item / Hq of this entry
  void *o2;       // optional second destination, row r -> o2 row o2_row0 + r
  int64_t o2_row0;
};

struct MergeLaunch {
  int32_t hq;
  int32_t n_entries;
  int32_t total_rows;
  MergeEntry e[kMaxEntries];
};

// Important-token selection: per-row scores over the selection layers, then a
// top-n per request (up to kMaxSelectReqs requests per top-n launch).
constexpr int kMaxSelectLayers = 8;
constexpr int kMaxSelectReqs = 64;
struct SelectReq {
  int64_t doc0;   // first score (document row) of the request
  int32_t L_d;    // document rows
  int32_t n;      // tokens to keep
  int32_t imp0;   // first output index slot (cu_imp[b])
};
struct SelectLaunch {
  const void *fresh[kMaxSelectLayers];   // [rows][Hkv][D] per layer
  const void *cached[kMaxSelectLayers];
  float *scores;                         // [rows]
  int32_t *idx;                          // [sum n]
  int64_t rows;
  int32_t row_bytes;                     // Hkv * D * element bytes, multiple of 16, <= 4096
  int32_t n_layers;
  int32_t n_req;
  SelectReq req[kMaxSelectReqs];
};
static_assert(sizeof(SelectLaunch) < 4096, "selection launch must fit 4 KiB of kernel arguments");

// Row movement (gather / scatter), byte copies in 16-byte units.
struct RowReq {
  int64_t base;     // token-row base of the request in the full-length buffer
  int32_t imp0;     // first important row / idx entry (cu_imp[b])
  int32_t n_imp;
  int32_t q0;       // first question row (cu_q[b])
  int32_t n_q;
  int32_t L_d;
};

struct RowLaunch {
  int32_t n_req;
  int32_t total_imp;  // sum of n_imp over these requests
  int32_t total_q;    // sum of n_q (scatter only)
  int32_t units;      // 16-byte units per row
  const int32_t *idx; // full idx array (entries indexed by imp0 + i)
  RowReq r[kMaxRowReqs];
};

struct ScatterPair {
  const void *src_imp;  // [.][row] rows by important index
  const void *src_q;    // [.][row] rows by question index
  void *dst;            // full-length token rows
};

// Kernel launchers (defined in attn.hip / rows.hip). Return the launch error.
// kernel names differ per stage so that profiles tell the stages apart
enum class AttnKind { kSelf = 0, kQdoc = 1 };
hipError_t launch_attention(int dtype, int head_dim, AttnKind kind,
                            const AttnLaunch &p, hipStream_t s);
hipError_t launch_attention_bf16(int head_dim, AttnKind kind, const AttnLaunch &p,
                                 hipStream_t s);
hipError_t launch_merge(int dtype, int head_dim, const MergeLaunch &p,
                        hipStream_t s);
// merge of the bf16 stage-2 split partials (attn_bf16.hip)
hipError_t launch_qdoc_merge_bf16(int head_dim, const MergeLaunch &p, hipStream_t s);
hipError_t launch_gather(const RowLaunch &p, int64_t src_base_unused,
                         const void *src, void *dst, hipStream_t s);
hipError_t launch_scatter(const RowLaunch &p, const ScatterPair *pairs,
                          int n_pairs, hipStream_t s);
hipError_t launch_check_indices(const RowLaunch &p, int32_t *d_bad,
                                int accumulate, hipStream_t s);
hipError_t launch_select_scores(const SelectLaunch &p, bool bf16, hipStream_t st);
hipError_t launch_select_topn(const SelectLaunch &p, hipStream_t st);

// ---- dense projections (C = A W^T + bias + residual, bf16) -------------------
struct GemmArgs {
  const void *A;         // [M][K]
  const void *W;         // [N][K]
  const void *bias;      // [N] or null
  const void *residual;  // [M][N] or null (may be C itself)
  void *C;               // [M][N]
  int64_t M;
  int32_t N, K;          // N % 128 == 0 (glu: N % 64 == 0), K % 64 == 0
  // glu: W is [2N][K], the gate rows then the up rows, and C[m][j] =
  // SiLU((A W^T)[m][j]) * (A W^T)[m][N + j] (no bias or residual)
  int32_t glu;
  int32_t tiles_m, tiles_n;  // filled by launch_gemm
  // launch_gemm_split only: output tiles t_begin .. t_begin + t_count - 1 of
  // the tile order; with `part` set each tile's k range is cut into k_parts
  // pieces whose fp32 sums go to part[(tile - t_begin) * k_parts + piece]
  // ([TM][TN] each) instead of C
  int32_t t_begin, t_count, k_parts;
  float *part;
};
hipError_t launch_gemm(const GemmArgs &a, hipStream_t st);
// The same product, with the output tiles that do not fill a whole round of
// the resident workgroups cut along k over the idle slots: their fp32 pieces
// go to `part` (at most part_bytes) and a reduction adds them, the bias and
// the residual. Falls back to launch_gemm when that does not apply (gated
// mode, too little workspace or k).
hipError_t launch_gemm_split(const GemmArgs &a, float *part, size_t part_bytes, hipStream_t st);
constexpr size_t kGemmPartBytes = (size_t)512 * 128 * 128 * 4;  // fp32 pieces of one round of small tiles
hipError_t launch_rmsnorm(int64_t rows, int width, const void *x, const void *w, float eps, void *y,
                          hipStream_t st);
hipError_t launch_rope(int64_t rows, int heads, int d, int64_t row_stride, void *x, const int32_t *pos,
                       double theta, hipStream_t st);
hipError_t launch_silu_mul(int64_t rows, int width, const void *gu, void *out, hipStream_t st);

}  // namespace daf
