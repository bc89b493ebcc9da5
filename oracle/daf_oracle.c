/*
 * Decoupled Attention Fusion (DAF): CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library. The product path (the
 * HIP library) shares no code, header or table with it and never calls it.
 *
 * Everything here is the plain definition of what the paper's method computes,
 * written naively: explicit materialised masks, a three-pass softmax, and
 * accumulation in double precision. Inputs are float32 values (for bfloat16
 * workloads, the exact bfloat16 values widened to float32), which are exactly
 * representable in double, so the oracle's own error is rounding of fp64 sums.
 *
 * Paper sections followed:
 *   - Sec. 2 item 1 (important-token selection & self-attention): the selected
 *     rows of every document are packed into one array, and each of them
 *     attends over keys from that array alone (the Complexity Analysis
 *     paragraph gives the same key set).
 *   - Sec. 2 item 2 (question-document self-attention): question rows attend
 *     over an L_q x (L_d + L_q) matrix whose keys are all preceding document
 *     tokens and the question itself, using the hybrid KV cache in which the
 *     important tokens' rows were already replaced by recomputed K/V.
 *   - Sec. 2 item 3 (state fusion): stage outputs are written into the hidden
 *     states.
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *   - stage-1 mask is causal by original position (decoder model);
 *   - stage-2 question-to-question part is causal, aligned to the bottom right;
 *   - softmax scale is a parameter (1/sqrt(head_dim) by default);
 *   - query head h reads key/value head floor(h / (Hq / Hkv)).
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC (see oracle/build.py). Compiling with
 * -DDAF_ORACLE_MUTANT=k plants mistake k; the test suite uses those builds to
 * show that the pins catch plausible errors. A normal build has no mutant.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifndef DAF_ORACLE_MUTANT
#define DAF_ORACLE_MUTANT 0
#endif

int daf_oracle_mutant(void) { return DAF_ORACLE_MUTANT; }

/* Threads the OpenMP loops of this library use. */
int daf_oracle_threads(void) { return omp_get_max_threads(); }

/* Row gather, byte for byte: dst[i] = src[rows[i]]  (the row collection of
 * Sec. 2 item 1). */
void daf_oracle_gather_rows(const uint8_t *src, int64_t row_bytes,
                            const int64_t *rows, int64_t nrows, uint8_t *dst) {
  int64_t count = nrows;
#if DAF_ORACLE_MUTANT == 8
  if (count > 0) count -= 1; /* planted: last row dropped */
#endif
  for (int64_t i = 0; i < count; ++i)
    memcpy(dst + i * row_bytes, src + rows[i] * row_bytes, (size_t)row_bytes);
}

/* Row scatter, byte for byte: dst[rows[i]] = src[i].  Used to build the hybrid
 * KV cache (Sec. 2 item 2) and to fuse stage outputs into the hidden states
 * (Sec. 2 item 3). */
void daf_oracle_scatter_rows(uint8_t *dst, int64_t row_bytes,
                             const int64_t *rows, int64_t nrows,
                             const uint8_t *src) {
  for (int64_t i = 0; i < nrows; ++i) {
    int64_t from = i;
#if DAF_ORACLE_MUTANT == 9
    from = nrows - 1 - i; /* planted: source rows reversed */
#endif
    memcpy(dst + rows[i] * row_bytes, src + from * row_bytes, (size_t)row_bytes);
  }
}

/* Stage-1 mask (Sec. 2 item 1 and the Complexity Analysis): query row r, at
 * original position pos[rows[r]], may see important token j iff token j does
 * not come after it in the original sequence. Keys are important tokens only.
 * mask is [nrows][n], 1 = visible. */
void daf_oracle_mask_stage1(const int64_t *pos, int64_t n, const int64_t *rows,
                            int64_t nrows, uint8_t *mask) {
  for (int64_t r = 0; r < nrows; ++r) {
    int64_t pi = pos[rows[r]];
    for (int64_t j = 0; j < n; ++j) {
#if DAF_ORACLE_MUTANT == 3
      /* planted: mask by condensed index instead of original position */
      mask[r * n + j] = (uint8_t)(j <= rows[r]);
#else
      mask[r * n + j] = (uint8_t)(pos[j] <= pi);
#endif
    }
  }
}

/* Stage-2 mask (Sec. 2 item 2): question row q (0-based within the question)
 * sees every document key 0..L_d-1 and the question keys L_d..L_d+q. mask is
 * [nrows][L_d + L_q], 1 = visible. */
void daf_oracle_mask_stage2(int64_t L_d, int64_t L_q, const int64_t *rows,
                            int64_t nrows, uint8_t *mask) {
  int64_t T = L_d + L_q;
  for (int64_t r = 0; r < nrows; ++r) {
    int64_t q = rows[r];
    for (int64_t k = 0; k < T; ++k) {
      int vis;
#if DAF_ORACLE_MUTANT == 4
      vis = 1; /* planted: question part not causal */
#elif DAF_ORACLE_MUTANT == 10
      vis = (k < L_d) || (k - L_d < q) || (k == 0); /* planted: own key dropped */
#else
      vis = (k < L_d) || (k - L_d <= q);
#endif
      mask[r * T + k] = (uint8_t)vis;
    }
  }
}

/* Position-causal mask for the comparison patterns (Complexity Analysis:
 * recomputation schemes in which the recomputed tokens and the question attend
 * over the full context). Query row r sits at original position qpos[rows[r]]
 * of a key sequence of nk tokens and sees keys 0..qpos. mask is [nrows][nk],
 * 1 = visible. With qpos[i] = i this is plain causal attention over the whole
 * sequence (full recomputation). */
void daf_oracle_mask_position(const int64_t *qpos, const int64_t *rows,
                              int64_t nrows, int64_t nk, uint8_t *mask) {
  for (int64_t r = 0; r < nrows; ++r) {
    int64_t p = qpos[rows[r]];
#if DAF_ORACLE_MUTANT == 12
    p += 1; /* planted: one key past the query's own position visible */
#endif
    for (int64_t k = 0; k < nk; ++k) mask[r * nk + k] = (uint8_t)(k <= p);
  }
}

/* Scaled dot-product attention with an explicit mask, by definition.
 *
 *   q: [nq][hq][d] float32 (only rows listed in `rows` are used)
 *   k, v: [nk][hkv][d] float32
 *   mask: [nrows][nk] uint8, row r belongs to query row rows[r]
 *   o: [nrows][hq][d] double, lse: [nrows][hq] double (natural log),
 *   p: optional [nrows][hq][nk] double, the probability matrix.
 *
 * For query head h the key/value head is g = floor(h / (hq / hkv)). Scores
 * s_j = scale * <q, k_j> over visible j; m = max s_j; w_j = exp(s_j - m);
 * l = sum w_j; o = sum (w_j / l) v_j; lse = m + ln l.
 * Returns -1 if some row has no visible key (never the case for DAF masks).
 */
int daf_oracle_masked_attention(const float *q, const float *k, const float *v,
                                const uint8_t *mask, int64_t nk, int32_t hq,
                                int32_t hkv, int32_t d, double scale,
                                const int64_t *rows, int64_t nrows, double *o,
                                double *lse, double *p) {
  const int32_t group = hq / hkv;
  int bad = 0;
#pragma omp parallel
  {
    double *s = (double *)malloc(sizeof(double) * (size_t)(nk > 0 ? nk : 1));
#pragma omp for schedule(dynamic, 1) reduction(| : bad)
    for (int64_t t = 0; t < nrows * (int64_t)hq; ++t) {
      const int64_t r = t / hq;
      const int32_t h = (int32_t)(t % hq);
#if DAF_ORACLE_MUTANT == 2
      const int32_t g = h % hkv; /* planted: interleaved GQA map */
#else
      const int32_t g = h / group;
#endif
      const float *qi = q + (rows[r] * hq + h) * (int64_t)d;
      const uint8_t *mr = mask + r * nk;
      double sc = scale;
#if DAF_ORACLE_MUTANT == 1
      sc = 1.0; /* planted: scale dropped */
#endif
      /* pass 1: scores and their maximum over visible keys */
      double m = -INFINITY;
      for (int64_t j = 0; j < nk; ++j) {
        if (!mr[j]) continue;
        const float *kj = k + (j * hkv + g) * (int64_t)d;
        double acc = 0.0;
        int32_t dd = d;
#if DAF_ORACLE_MUTANT == 11
        dd = d - 1; /* planted: last feature dropped from the dot product */
#endif
        for (int32_t c = 0; c < dd; ++c) acc += (double)qi[c] * (double)kj[c];
        s[j] = sc * acc;
        if (s[j] > m) m = s[j];
      }
      if (m == -INFINITY) {
        bad |= 1;
        continue;
      }
      /* pass 2: exponentials and their sum */
      double l = 0.0;
      int64_t last_visible = -1;
      for (int64_t j = 0; j < nk; ++j) {
        if (!mr[j]) continue;
        s[j] = exp(s[j] - m);
        last_visible = j;
      }
      for (int64_t j = 0; j < nk; ++j) {
        if (!mr[j]) continue;
#if DAF_ORACLE_MUTANT == 7
        if (j == last_visible && j != 0) continue; /* planted: term dropped from l */
#endif
        l += s[j];
      }
      (void)last_visible;
      /* pass 3: normalised weights times values */
      double *oi = o + (r * hq + h) * (int64_t)d;
      for (int32_t c = 0; c < d; ++c) oi[c] = 0.0;
      for (int64_t j = 0; j < nk; ++j) {
        if (!mr[j]) continue;
        const double w = s[j] / l;
#if DAF_ORACLE_MUTANT == 5
        const float *vj = k + (j * hkv + g) * (int64_t)d; /* planted: K used as V */
#else
        const float *vj = v + (j * hkv + g) * (int64_t)d;
#endif
        for (int32_t c = 0; c < d; ++c) oi[c] += w * (double)vj[c];
      }
#if DAF_ORACLE_MUTANT == 6
      lse[r * hq + h] = log(l); /* planted: max term missing from lse */
#else
      lse[r * hq + h] = m + log(l);
#endif
      if (p) {
        double *pi = p + (r * hq + h) * nk;
        for (int64_t j = 0; j < nk; ++j) pi[j] = mr[j] ? s[j] / l : 0.0;
      }
    }
    free(s);
  }
  return bad ? -1 : 0;
}
