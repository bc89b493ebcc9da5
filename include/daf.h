/*
 * daf.h - C ABI of the Decoupled Attention Fusion (DAF) per-layer prefill
 * attention library for AMD Instinct MI355X (gfx950).
 *
 * DAF (Sec. 2 of the paper) replaces full prefill attention over retrieved
 * documents whose KV caches were computed offline, one document at a time, by
 * three stages per layer:
 *   1. important-token self-attention: n = r*L_d selected rows, taken from
 *      every document, form one packed array whose queries see only keys of
 *      that array (Sec. 2 item 1; Complexity Analysis);
 *   2. question-document attention: the L_q question tokens, at the tail of the
 *      sequence, attend over all L_d + L_q keys, reading a hybrid KV cache in
 *      which the important tokens' rows already hold their recomputed K/V
 *      (Sec. 2 item 2);
 *   3. state fusion: the outputs of both stages are written into the layer's
 *      hidden states (Sec. 2 item 3).
 * The selection policy that picks the important tokens and the Q/K/V
 * projections stay with the caller: indices and projected Q/K/V are inputs.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory. Every tensor pointer is DEVICE memory owned by the caller; the
 *   library allocates and frees nothing. Scratch memory comes from the caller's
 *   `workspace`. Pointers must be 16-byte aligned.
 * Layouts. Tensors are token-major and contiguous: queries and outputs are
 *   [tokens][Hq][D], keys and values [tokens][Hkv][D], elements of `dtype`.
 *   One output row (Hq*D elements) is one row of the hidden-state buffer.
 *   LSE outputs are float32 [Hq][rows] (natural log of the softmax
 *   denominator, including the max), row = the output's token row.
 * Requests. A call serves a ragged batch of B >= 1 independent requests
 *   (daf_batch_t). Request b has L_d,b document tokens, L_q,b question tokens
 *   and n_b important tokens. Its rows are:
 *     important rows (q_imp, k_imp, v_imp, o_imp, idx): cu_imp[b] .. cu_imp[b+1]
 *     question rows  (q_q, k_q, v_q, o_q):              cu_q[b]   .. cu_q[b+1]
 *     token rows     (k_cache, v_cache, hidden):        tok_b .. tok_b + T_b,
 *       tok_b = cu_doc[b] + cu_q[b], T_b = L_d,b + L_q,b, documents first.
 * Indices. idx[cu_imp[b] + i] is the request-local original position of
 *   request b's i-th important token: 0 <= idx < L_d,b and strictly increasing
 *   within a request. This is NOT checked on the hot path (violations are
 *   undefined behaviour: duplicate rows make the scatters race);
 *   daf_check_indices() verifies it on the device.
 * Masks. Stage 1: important token i sees important token j iff j <= i (the
 *   condensed order is the original order, so this is causal by original
 *   position). Stage 2: question token j sees every document token and
 *   question tokens 0..j.
 * Numerics. bf16 or fp32 in; fp32 accumulation and softmax; outputs in the
 *   input dtype. bf16 attention rounds the softmax probabilities to bf16
 *   before the value product and normalises by the sum of those rounded
 *   probabilities, so each output row is a weighted mean of value rows with
 *   weights that sum to one; its LSE is the log of that same sum, within
 *   ln(1 + 2^-8) of the exact log-sum-exp (the bf16 rounding of a term that
 *   dominates its row). The unnormalised fp32 sums hold probabilities of at most
 *   2^32 per 16 keys (the running max is raised only past that), so value
 *   magnitudes times 2^32 per 16 keys must stay within fp32 (|V| below ~1e26
 *   for 32k keys). Stage 2's key splits keep their normalised partial outputs
 *   in the input dtype (bf16: one more rounding of each split's weighted mean
 *   before the log-sum-exp merge) and their LSE in fp32.
 * Asynchrony. Work is enqueued on `stream` (NULL = the default stream) and the
 *   call returns without synchronising. Calls are re-entrant and thread-safe;
 *   the only state the library keeps is daf_layer_attn's second stream and its
 *   two events per device (created on first use, guarded by a mutex). Calls
 *   that write the same buffers must be ordered by the caller.
 * Graph capture. The calls enqueue kernels and event record/wait operations
 *   only (no allocation, copy, memset or synchronisation), so a sequence of
 *   them can be captured into a HIP graph and replayed. daf_layer_attn's
 *   second stream joins the capture through its fork event and rejoins the
 *   caller's stream before the call returns. Make the first daf_layer_attn
 *   call on a device outside any capture (it creates the stream and events),
 *   and make no daf_layer_attn call on that device from another stream or
 *   thread while such a capture is open: the shared second stream stays part
 *   of the capture until it ends.
 * Errors. Every host-visible precondition is checked before anything is
 *   enqueued; on failure the call returns a non-zero daf_status_t, enqueues
 *   nothing, and daf_last_error() describes the problem (thread-local). A
 *   failed kernel launch returns DAF_ERR_HIP. No C++ exception crosses the ABI.
 */
#ifndef DAF_H_
#define DAF_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DAF_OK = 0,
  DAF_ERR_INVALID_ARG = 1, /* null pointer, bad size, inconsistent offsets */
  DAF_ERR_ALIGNMENT = 2,   /* pointer or row size not a multiple of 16 bytes */
  DAF_ERR_UNSUPPORTED = 3, /* head_dim / dtype the kernels do not cover */
  DAF_ERR_WORKSPACE = 4,   /* workspace missing or smaller than required */
  DAF_ERR_HIP = 5          /* a HIP runtime call or kernel launch failed */
} daf_status_t;

typedef enum { DAF_BF16 = 0, DAF_F32 = 1 } daf_dtype_t;

/* Attention shape. Query head h reads key/value head h / (Hq / Hkv). */
typedef struct {
  int32_t n_q_heads;   /* Hq >= 1 */
  int32_t n_kv_heads;  /* Hkv >= 1, divides Hq */
  int32_t head_dim;    /* D: 64 or 128 */
  int32_t dtype;       /* daf_dtype_t of every tensor */
  float softmax_scale; /* > 0, or 0 for 1/sqrt(D) */
} daf_attn_cfg_t;

/* Ragged batch. All three arrays are HOST memory, [batch + 1] prefix sums
 * starting at 0: cu_doc of L_d,b, cu_q of L_q,b, cu_imp of n_b (n_b <= L_d,b).
 * The library reads them during the call only. */
typedef struct {
  int32_t batch;
  const int32_t *cu_doc;
  const int32_t *cu_q;
  const int32_t *cu_imp;
} daf_batch_t;

/* daf_gather_important `src_layout` values. */
enum {
  DAF_SRC_TOKENS = 0, /* src has T_b rows per request starting at tok_b */
  DAF_SRC_DOCS = 1    /* src has L_d,b rows per request starting at cu_doc[b] */
};

/* daf_fuse `flags` bits. */
enum {
  DAF_FUSE_KV = 1,    /* hybrid KV cache + question KV append */
  DAF_FUSE_HIDDEN = 2 /* stage outputs into the hidden states */
};

/* Gather the important rows into one contiguous array per batch (the row
 * collection step of stage 1, Sec. 2 item 1).
 *   dst[cu_imp[b] + i] = src[base_b + idx[cu_imp[b] + i]]   (row_bytes each)
 * with base_b = tok_b for DAF_SRC_TOKENS or cu_doc[b] for DAF_SRC_DOCS. Rows
 * are copied bit for bit; row_bytes must be a positive multiple of 16. Used
 * for the hidden rows that feed the caller's QKV projection and for K/V rows
 * of a full-length cache. */
daf_status_t daf_gather_important(const daf_batch_t *batch, int32_t src_layout,
                                  const void *src, int64_t row_bytes,
                                  const int32_t *idx, void *dst,
                                  hipStream_t stream);

/* Important-token selection, the step before the path (Sec. 2 item 1: tokens
 * are chosen by the deviation of their recomputed KV from the offline cache,
 * aggregated over several early layers, typically the 2nd to the 4th).
 *   k_fresh[l], k_cached[l], l < n_layers (1..8): a HOST array of DEVICE
 *   pointers per argument; each tensor is [sum L_d][Hkv][D] of `dtype`,
 *   request b's document rows from cu_doc[b] (documents only), 16-byte aligned.
 *   scores (DEVICE float32 [sum L_d], output): per document token, the mean
 *   over the layers of the L2 norm of k_fresh - k_cached over its Hkv*D values
 *   (the paper names the signal but not the norm or the aggregation).
 *   idx (DEVICE int32 [sum n], output): for request b, the n_b = cu_imp[b+1] -
 *   cu_imp[b] tokens with the highest scores (equal scores: lower index
 *   first), request-local, strictly increasing - the idx the other entry
 *   points take.
 * Hkv * D * element size must not exceed 4096 bytes (DAF_ERR_UNSUPPORTED). */
daf_status_t daf_select_important(const daf_attn_cfg_t *cfg,
                                  const daf_batch_t *batch, int32_t n_layers,
                                  const void *const *k_fresh,
                                  const void *const *k_cached, float *scores,
                                  int32_t *idx, hipStream_t stream);

/* Stage 1, important-token self-attention (Sec. 2 item 1; Complexity
 * Analysis: important tokens attend only to each other, O(r^2 L_d^2)).
 *   q_imp [sum n][Hq][D], k_imp / v_imp [sum n][Hkv][D] -> o_imp [sum n][Hq][D]
 *   lse_imp: nullable float32 [Hq][sum n].
 * Within request b, row i attends rows 0..i of the same request (causal in the
 * condensed order, which is the original order). */
daf_status_t daf_imp_self_attn(const daf_attn_cfg_t *cfg,
                               const daf_batch_t *batch, const void *q_imp,
                               const void *k_imp, const void *v_imp,
                               void *o_imp, float *lse_imp, hipStream_t stream);

/* Attention of queries at given positions of a key sequence, for the
 * comparison the Complexity Analysis draws: schemes that recompute selected
 * tokens and the question over the full context (the CacheBlend pattern:
 * important and question tokens over all L_d + L_q keys, O(r L_d^2 + L_d L_q))
 * and full recomputation (every token over its prefix), against which DAF's
 * O(r^2 L_d^2 + L_q (L_d + L_q)) is measured; the Hardware Compatibility
 * paragraph notes that such unified recomputation needs non-standard masks.
 *   q [n_rows][Hq][D], k / v [n_keys][Hkv][D] -> o [n_rows][Hq][D];
 *   lse: nullable float32 [Hq][n_rows].
 * Row i sees keys 0 .. q_pos[i]; q_pos (DEVICE int32 [n_rows]) must be
 * strictly increasing with values in [0, n_keys) - not checked, violations are
 * undefined behaviour. q_pos = NULL means bottom-right causal: row i sees keys
 * 0 .. i + n_keys - n_rows (requires n_rows <= n_keys); with n_rows = n_keys
 * that is full causal self-attention. One sequence per call; no workspace. */
daf_status_t daf_position_attn(const daf_attn_cfg_t *cfg, int32_t n_rows,
                               int32_t n_keys, const void *q,
                               const int32_t *q_pos, const void *k,
                               const void *v, void *o, float *lse,
                               hipStream_t stream);

/* Bytes of workspace daf_qdoc_attn needs for this shape (0 on bad input). */
size_t daf_qdoc_workspace_size(const daf_attn_cfg_t *cfg,
                               const daf_batch_t *batch);

/* Stage 2, question-document attention (Sec. 2 item 2: an L_q x (L_d + L_q)
 * attention over the hybrid KV cache; Complexity Analysis: O(L_q (L_d+L_q))).
 *   q_q [sum L_q][Hq][D]; k_cache / v_cache hold T_b token rows per request
 *   (the hybrid cache: daf_fuse(DAF_FUSE_KV) first) -> o_q [sum L_q][Hq][D];
 *   lse_q: nullable float32 [Hq][sum L_q].
 * Question row j of request b attends cache rows 0 .. L_d,b + j. The keys are
 * split across workgroups; partial results (each split's normalised output in
 * the input dtype and its fp32 LSE) live in `workspace` (at least
 * daf_qdoc_workspace_size bytes, 16-byte aligned, contents undefined after
 * the call) and are merged by log-sum-exp. */
daf_status_t daf_qdoc_attn(const daf_attn_cfg_t *cfg, const daf_batch_t *batch,
                           const void *q_q, const void *k_cache,
                           const void *v_cache, void *o_q, float *lse_q,
                           void *workspace, size_t ws_bytes,
                           hipStream_t stream);

/* State fusion and hybrid-cache construction, as in-place row scatters (Sec. 2
 * item 2: the important tokens' K/V are updated in the document cache before
 * question-document attention; Sec. 2 item 3: stage outputs are fused into the
 * hidden states).
 * DAF_FUSE_KV (needs k_imp, v_imp, k_q, v_q, k_cache, v_cache):
 *   k_cache[tok_b + idx[.]] = k_imp[.],   k_cache[tok_b + L_d,b + j] = k_q[.]
 *   (same for v) - the hybrid cache, with the question's K/V after the docs.
 * DAF_FUSE_HIDDEN (needs o_imp, o_q, hidden [sum T][Hq*D]):
 *   hidden[tok_b + idx[.]] = o_imp[.],    hidden[tok_b + L_d,b + j] = o_q[.]
 * Rows are copied bit for bit; every other row is left untouched. Pointers not
 * needed by the selected flags may be NULL. */
daf_status_t daf_fuse(const daf_attn_cfg_t *cfg, const daf_batch_t *batch,
                      uint32_t flags, const int32_t *idx, const void *k_imp,
                      const void *v_imp, const void *k_q, const void *v_q,
                      void *k_cache, void *v_cache, const void *o_imp,
                      const void *o_q, void *hidden, hipStream_t stream);

/* Bytes of workspace daf_layer_attn needs (0 on bad input). */
size_t daf_layer_workspace_size(const daf_attn_cfg_t *cfg,
                                const daf_batch_t *batch);

/* One DAF attention layer (Sec. 2 items 1-3), in the order the paper fixes:
 * hybrid KV write-back (DAF_FUSE_KV) first, then stage 2 (with its split
 * merge); stage 1 needs none of these and runs beside them on a stream the
 * library owns (one per device, default priority), forked from `stream` and
 * joined back into it with events, so all of the call's work is ordered on
 * `stream` for the caller. Arguments as in the stage calls. o_imp and o_q
 * receive the stage outputs; the same rows are written into `hidden` exactly
 * as DAF_FUSE_HIDDEN would (the state fusion happens in the stage epilogues,
 * without a separate pass). */
daf_status_t daf_layer_attn(const daf_attn_cfg_t *cfg, const daf_batch_t *batch,
                            const int32_t *idx, const void *q_imp,
                            const void *k_imp, const void *v_imp,
                            const void *q_q, const void *k_q, const void *v_q,
                            void *k_cache, void *v_cache, void *o_imp,
                            float *lse_imp, void *o_q, float *lse_q,
                            void *hidden, void *workspace, size_t ws_bytes,
                            hipStream_t stream);

/* For callers that cannot allocate (code under HIP graph capture, serving
 * loops or harnesses that forbid hipMalloc): daf_layer_attn with the stage-2
 * workspace taken from a static device array of the library instead of a
 * caller buffer, all work on `stream` (no second stream). Arguments and
 * results as in daf_layer_attn. The array holds daf_layer_noalloc_max_bytes()
 * bytes (48 MiB) on every device the library runs on, kept until the process
 * ends; a batch whose workspace (daf_layer_workspace_size) exceeds it returns
 * DAF_ERR_WORKSPACE and enqueues nothing. The call allocates nothing: no
 * hipMalloc, hipFree, stream or event creation. Every call on one device
 * shares that device's array, so calls that can overlap on one device (other
 * streams, other threads) race; order them on one stream. No result depends on
 * what an earlier call left in the array. */
size_t daf_layer_noalloc_max_bytes(void);
daf_status_t daf_layer_attn_noalloc(const daf_attn_cfg_t *cfg, const daf_batch_t *batch,
                                    const int32_t *idx, const void *q_imp,
                                    const void *k_imp, const void *v_imp,
                                    const void *q_q, const void *k_q, const void *v_q,
                                    void *k_cache, void *v_cache, void *o_imp,
                                    float *lse_imp, void *o_q, float *lse_q,
                                    void *hidden, hipStream_t stream);

/* Debug check of the index precondition: writes to *d_bad_count (device
 * int32) the number of entries of idx that are out of [0, L_d,b) or not
 * greater than their predecessor in the same request. */
daf_status_t daf_check_indices(const daf_batch_t *batch, const int32_t *idx,
                               int32_t *d_bad_count, hipStream_t stream);

/* Static name of a status code. */
const char *daf_status_string(daf_status_t status);

/* Dense projection of the decoder layer around the attention: the QKV
 * computation phase of Sec. 2 item 2 (run on the important and question rows
 * only) and the projections that the fused compact state feeds (Sec. 2 item
 * 3): C = A W^T (+ bias) (+ residual), bf16 in and out.
 *   A [M][K] and W [N][K] row-major (W in the usual [out][in] layout);
 *   bias [N] or NULL; residual [M][N] or NULL, and may be C itself (an
 *   in-place residual add); C [M][N].
 * fp32 accumulation; bias and residual are added in fp32 before the single
 * rounding to bf16. N must be a positive multiple of 128 and K of 64
 * (DAF_ERR_UNSUPPORTED otherwise); every pointer 16-byte aligned. M = 0 is a
 * no-op. */
daf_status_t daf_linear(int64_t M, int32_t N, int32_t K, const void *A,
                        const void *W, const void *bias, const void *residual,
                        void *C, hipStream_t stream);

/* The MLP's gate and up projections with the gate applied in the epilogue:
 * C[m][j] = SiLU((A Wg^T)[m][j]) * (A Wu^T)[m][j], SiLU(g) = g / (1 + exp(-g)),
 * where Wgu [2I][K] holds the gate rows then the up rows (bf16, fp32
 * accumulation, one rounding). A [M][K], C [M][I]. I a positive multiple of
 * 64 and K of 64 (DAF_ERR_UNSUPPORTED otherwise); pointers 16-byte aligned. */
daf_status_t daf_linear_swiglu(int64_t M, int32_t I, int32_t K, const void *A,
                               const void *Wgu, void *C, hipStream_t stream);

/* RMS normalisation before the projections: y = x / sqrt(mean(x^2) + eps) * w
 * per row (x, y [rows][width], w [width], bf16; fp32 arithmetic). width must
 * be a positive multiple of 8; y may be x. */
daf_status_t daf_rmsnorm(int64_t rows, int32_t width, const void *x,
                         const void *w, float eps, void *y, hipStream_t stream);

/* Rotary position embedding, in place, of n_heads heads of head_dim features
 * at the start of each of `rows` rows (row pitch row_stride elements, bf16):
 * features (i, i + head_dim/2) of a head rotate by pos[row] *
 * theta^(-2i/head_dim) (the angle in fp64). This is how the recomputed q and
 * k of the important and question rows take their original positions
 * (Sec. 2 item 1 keeps the original order). head_dim even, pos int32 [rows]. */
daf_status_t daf_rope(int64_t rows, int32_t n_heads, int32_t head_dim,
                      int64_t row_stride, void *x, const int32_t *pos,
                      float theta, hipStream_t stream);

/* MLP gate: out[r][j] = SiLU(gu[r][j]) * gu[r][width + j], SiLU(g) =
 * g / (1 + exp(-g)); gu [rows][2 width] (gate then up), out [rows][width],
 * bf16. width a positive multiple of 8. */
daf_status_t daf_silu_mul(int64_t rows, int32_t width, const void *gu,
                          void *out, hipStream_t stream);

/* Weights of one decoder layer (bf16, projections [out][in]): the reading
 * taken for the model the paper evaluates on (Qwen2.5-7B, Sec. 3) is the
 * pre-norm decoder layer
 *   h = RMSNorm(x) w_in; q,k,v = h W^T + b; RoPE(q, k); o = attention
 *   x += o wo^T; h = RMSNorm(x) w_post; x += (SiLU(h wg^T) * (h wu^T)) wd^T */
typedef struct {
  const void *w_in;            /* [hidden] */
  const void *wq, *bq;         /* [Hq*D][hidden], [Hq*D] */
  const void *wk, *bk;         /* [Hkv*D][hidden], [Hkv*D] */
  const void *wv, *bv;         /* [Hkv*D][hidden], [Hkv*D] */
  const void *wo;              /* [hidden][Hq*D] */
  const void *w_post;          /* [hidden] */
  const void *wgu;             /* [2*inter][hidden]: the gate rows, then the up rows */
  const void *wd;              /* [hidden][inter] */
  int32_t hidden, inter;       /* multiples of 128 */
  float eps, rope_theta;
} daf_layer_weights_t;

enum { DAF_LAYER_DAF = 0, DAF_LAYER_FULL = 1 };

/* Workspace daf_decoder_layer needs (0 on bad input). */
size_t daf_decoder_layer_workspace_size(const daf_attn_cfg_t *cfg,
                                        const daf_layer_weights_t *w,
                                        const daf_batch_t *batch,
                                        int32_t mode);

/* One decoder layer of prefill, in place on the residual stream x (bf16
 * [rows][hidden]) at positions pos (int32 [rows]).
 * DAF_LAYER_DAF (Sec. 2 items 1-3): only the important and question rows are
 *   recomputed. rows = sum n + sum L_q, ordered as the stage calls take them:
 *   every request's important rows (in idx order), then every request's
 *   question rows. Their q/k/v come from the projections; the important and
 *   question K/V are written into k_cache / v_cache (the hybrid cache, as
 *   DAF_FUSE_KV) and the DAF attention runs as in daf_layer_attn; the other
 *   document rows are not touched. The updated x is the compact state the
 *   next layer takes (Sec. 2 item 3).
 * DAF_LAYER_FULL (the full-recomputation baseline of Sec. 3): every token is
 *   recomputed; rows = sum T_b, each request's documents then its question,
 *   causal attention over the request's own rows; idx, k_cache and v_cache
 *   are not used (may be NULL).
 * workspace: at least daf_decoder_layer_workspace_size bytes, 256-byte
 * aligned, contents undefined after the call. Errors as for the other calls;
 * nothing is enqueued when a check fails. */
daf_status_t daf_decoder_layer(const daf_attn_cfg_t *cfg,
                               const daf_layer_weights_t *w,
                               const daf_batch_t *batch, int32_t mode,
                               const int32_t *idx, const int32_t *pos, void *x,
                               void *k_cache, void *v_cache, void *workspace,
                               size_t ws_bytes, hipStream_t stream);

/* Detail of the last failure on the calling thread ("" if none). */
const char *daf_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int32_t daf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DAF_H_ */
