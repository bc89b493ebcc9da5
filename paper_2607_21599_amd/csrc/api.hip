// DAF C ABI: argument validation, launch planning and the one-layer driver.
// Every check runs on the host before anything is enqueued; the kernels live
// in attn.hip and rows.hip.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "daf.h"
#include "daf_internal.h"

namespace {

using namespace daf;

thread_local char g_err[512] = "";

daf_status_t fail(daf_status_t st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

daf_status_t ok() {
  g_err[0] = '\0';
  return DAF_OK;
}

daf_status_t hip_fail(hipError_t e, const char *what) {
  return fail(DAF_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

struct Cfg {
  int hq, hkv, group, d, dtype;
  float scale;
  int elem;    // bytes per element
  int key_tile;
};

struct Req {
  int L_d, L_q, n;
  int imp0, q0;
  int64_t tok0;  // first token row (cache / hidden)
};

struct Batch {
  std::vector<Req> r;
  int64_t total_imp = 0, total_q = 0, total_tok = 0;
};

daf_status_t parse_cfg(const daf_attn_cfg_t *c, Cfg &out) {
  if (!c) return fail(DAF_ERR_INVALID_ARG, "cfg is NULL");
  if (c->n_q_heads < 1 || c->n_kv_heads < 1)
    return fail(DAF_ERR_INVALID_ARG, "head counts must be >= 1 (Hq=%d, Hkv=%d)", c->n_q_heads,
                c->n_kv_heads);
  if (c->n_q_heads % c->n_kv_heads != 0)
    return fail(DAF_ERR_INVALID_ARG, "Hq=%d is not a multiple of Hkv=%d", c->n_q_heads, c->n_kv_heads);
  if (c->n_q_heads > 1024) return fail(DAF_ERR_UNSUPPORTED, "Hq=%d exceeds 1024", c->n_q_heads);
  if (c->head_dim != 64 && c->head_dim != 128)
    return fail(DAF_ERR_UNSUPPORTED, "head_dim=%d (supported: 64, 128)", c->head_dim);
  if (c->dtype != DAF_BF16 && c->dtype != DAF_F32)
    return fail(DAF_ERR_UNSUPPORTED, "dtype=%d (supported: DAF_BF16, DAF_F32)", c->dtype);
  if (!(c->softmax_scale >= 0.f) || !isfinite(c->softmax_scale))
    return fail(DAF_ERR_INVALID_ARG, "softmax_scale must be finite and >= 0");
  out.hq = c->n_q_heads;
  out.hkv = c->n_kv_heads;
  out.group = out.hq / out.hkv;
  out.d = c->head_dim;
  out.dtype = c->dtype;
  out.scale = c->softmax_scale > 0.f ? c->softmax_scale : 1.f / sqrtf((float)c->head_dim);
  out.elem = c->dtype == DAF_BF16 ? 2 : 4;
  out.key_tile = c->dtype == DAF_BF16 ? 64 : 32;
  return DAF_OK;
}

daf_status_t parse_batch(const daf_batch_t *b, Batch &out) {
  if (!b) return fail(DAF_ERR_INVALID_ARG, "batch is NULL");
  if (b->batch < 1) return fail(DAF_ERR_INVALID_ARG, "batch=%d must be >= 1", b->batch);
  if (!b->cu_doc || !b->cu_q || !b->cu_imp)
    return fail(DAF_ERR_INVALID_ARG, "cu_doc, cu_q and cu_imp must be non-NULL host arrays");
  if (b->cu_doc[0] != 0 || b->cu_q[0] != 0 || b->cu_imp[0] != 0)
    return fail(DAF_ERR_INVALID_ARG, "prefix arrays must start at 0");
  out.r.resize(b->batch);
  int64_t tok = 0;
  for (int i = 0; i < b->batch; ++i) {
    Req &q = out.r[i];
    // differences in 64 bits: a decreasing pair of int32 entries must not wrap
    const int64_t L_d = (int64_t)b->cu_doc[i + 1] - b->cu_doc[i];
    const int64_t L_q = (int64_t)b->cu_q[i + 1] - b->cu_q[i];
    const int64_t n = (int64_t)b->cu_imp[i + 1] - b->cu_imp[i];
    if (L_d < 0 || L_q < 0 || n < 0)
      return fail(DAF_ERR_INVALID_ARG, "request %d: prefix arrays must be non-decreasing", i);
    q.L_d = (int)L_d;  // each lies between 0 and INT32_MAX: the arrays start at 0 and do not decrease
    q.L_q = (int)L_q;
    q.n = (int)n;
    if (q.n > q.L_d)
      return fail(DAF_ERR_INVALID_ARG, "request %d: n=%d important tokens exceed L_d=%d", i, q.n, q.L_d);
    q.imp0 = b->cu_imp[i];
    q.q0 = b->cu_q[i];
    q.tok0 = tok;
    tok += (int64_t)q.L_d + q.L_q;
  }
  if (tok > INT32_MAX) return fail(DAF_ERR_UNSUPPORTED, "total token rows %lld exceed 2^31-1", (long long)tok);
  out.total_imp = b->cu_imp[b->batch];
  out.total_q = b->cu_q[b->batch];
  out.total_tok = tok;
  return DAF_OK;
}

// The attention kernels address one request's K/V rows through buffer
// descriptors with 32-bit byte offsets.
daf_status_t check_kv_extent(const Cfg &c, const Batch &b) {
  const int64_t row = (int64_t)c.hkv * c.d * c.elem;
  for (size_t i = 0; i < b.r.size(); ++i) {
    const int64_t t = (int64_t)b.r[i].L_d + b.r[i].L_q;
    if (t * row > INT32_MAX)
      return fail(DAF_ERR_UNSUPPORTED, "request %zu: %lld K/V bytes exceed 2 GiB per request", i,
                  (long long)(t * row));
  }
  return DAF_OK;
}

daf_status_t need_ptr(const void *p, const char *name) {
  if (!p) return fail(DAF_ERR_INVALID_ARG, "%s is NULL", name);
  if (reinterpret_cast<uintptr_t>(p) % 16 != 0)
    return fail(DAF_ERR_ALIGNMENT, "%s is not 16-byte aligned", name);
  return DAF_OK;
}

#define CHECK(expr)                   \
  do {                                \
    daf_status_t st_ = (expr);        \
    if (st_ != DAF_OK) return st_;    \
  } while (0)

// ---- stage-2 split plan (depends on the shape only) --------------------------
struct Split {
  int n_splits, split_keys;
};

// The bf16 split-key kernel packs (query head, 32-row block) units of a KV
// group four to a workgroup; the fp32 kernel runs one head per workgroup.
bool packed_qdoc(const Cfg &c) { return c.dtype == DAF_BF16; }
// workgroups per KV head and key split for a question of L_q rows
int qdoc_blocks(const Cfg &c, int L_q) {
  if (!packed_qdoc(c)) return (L_q + kAttnBM - 1) / kAttnBM;
  const int units = c.group * ((L_q + 31) / 32);
  return (units + 3) / 4;
}

std::vector<Split> plan_splits(const Cfg &c, const Batch &b) {
  const int BN = c.key_tile;
  double work = 0;
  for (const Req &q : b.r) {
    if (q.L_q == 0) continue;
    const int kbs = (q.L_d + q.L_q + BN - 1) / BN;
    // workgroups per split times key tiles
    const int wgs = packed_qdoc(c) ? c.hkv * qdoc_blocks(c, q.L_q) : c.hq * qdoc_blocks(c, q.L_q);
    work += (double)wgs * kbs;
  }
  const double per_wg = std::max(1.0, work / kTargetWorkgroups);
  std::vector<Split> out(b.r.size());
  for (size_t i = 0; i < b.r.size(); ++i) {
    const Req &q = b.r[i];
    const int kbs = std::max(1, (q.L_d + q.L_q + BN - 1) / BN);
    int s = (int)std::lround(kbs / per_wg);
    s = std::min(std::max(s, 1), kbs);
    const int blocks = (kbs + s - 1) / s;
    out[i].split_keys = blocks * BN;
    out[i].n_splits = (kbs + blocks - 1) / blocks;
  }
  return out;
}

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct WsLayout {
  size_t part_o_bytes, part_lse_bytes, total;
  int64_t part_rows;  // sum over requests of L_q * n_splits
};

WsLayout ws_layout(const Cfg &c, const Batch &b, const std::vector<Split> &sp) {
  WsLayout w{};
  w.part_rows = 0;
  for (size_t i = 0; i < b.r.size(); ++i) w.part_rows += (int64_t)b.r[i].L_q * sp[i].n_splits;
  // partial outputs in the input dtype (normalised, so bf16 keeps their precision
  // relative to the values), their LSE in fp32
  w.part_o_bytes = align_up((size_t)w.part_rows * c.hq * c.d * c.elem);
  w.part_lse_bytes = align_up((size_t)w.part_rows * c.hq * sizeof(float));
  w.total = w.part_o_bytes + w.part_lse_bytes;
  return w;
}

// ---- second stream for the layer call ----------------------------------------
// daf_layer_attn runs stage 1 on a library-owned stream (default priority),
// forked from and joined back into the caller's stream by events, so that it
// overlaps the KV write-back, stage 2 and the merge. One stream and two events
// per device, created on first use; the mutex keeps each call's fork and join
// together when several threads enqueue at once.
struct AuxStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
  bool tried = false, ok = false;
};
constexpr int kMaxDevices = 64;
std::mutex g_aux_mu;
AuxStream g_aux[kMaxDevices];

// the current device's stream, or null (then the call runs on one stream);
// call with g_aux_mu held
AuxStream *aux_stream() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  AuxStream &a = g_aux[dev];
  if (!a.tried) {
    a.tried = true;
    a.ok = hipStreamCreateWithFlags(&a.s, hipStreamNonBlocking) == hipSuccess &&
           hipEventCreateWithFlags(&a.fork, hipEventDisableTiming) == hipSuccess &&
           hipEventCreateWithFlags(&a.join, hipEventDisableTiming) == hipSuccess;
  }
  return a.ok ? &a : nullptr;
}

// ---- static scratch for the allocation-free layer call ------------------------
// daf_layer_attn_noalloc takes its stage-2 workspace from this array instead of
// a caller buffer. In host code `scratch` names a host-side stand-in, never the
// device memory: its device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// passed to kernels.
constexpr size_t kScratchBytes = (size_t)48 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchAddr {
  void *ptr = nullptr;
  bool tried = false;
  hipError_t err = hipSuccess;
};
std::mutex g_scratch_mu;
ScratchAddr g_scratch[kMaxDevices];

// the current device's scratch address, or null with `err` set
void *scratch_ptr(hipError_t &err) {
  int dev = -1;
  err = hipGetDevice(&dev);
  if (err != hipSuccess) return nullptr;
  if (dev < 0 || dev >= kMaxDevices) {
    err = hipErrorInvalidDevice;
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  ScratchAddr &a = g_scratch[dev];
  if (!a.tried) {
    a.tried = true;
    void *p = nullptr;
    a.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (a.err == hipSuccess) a.ptr = p;
  }
  err = a.err;
  return a.ptr;
}

// ---- attention work tables ----------------------------------------------------
AttnEntry self_entry(const Cfg &c, const Req &q, int64_t total_imp, const void *q_imp,
                     const void *k_imp, const void *v_imp, void *o_imp, float *lse_imp) {
  AttnEntry e{};
  const size_t qrow = (size_t)c.hq * c.d * c.elem, krow = (size_t)c.hkv * c.d * c.elem;
  e.q = static_cast<const char *>(q_imp) + q.imp0 * qrow;
  e.k = static_cast<const char *>(k_imp) + q.imp0 * krow;
  e.v = static_cast<const char *>(v_imp) + q.imp0 * krow;
  e.o = static_cast<char *>(o_imp) + q.imp0 * qrow;
  e.lse = lse_imp ? lse_imp + q.imp0 : nullptr;
  e.lse_stride = (int32_t)total_imp;
  e.n_rows = q.n;
  e.n_keys = q.n;
  const int mbs = (q.n + kAttnBM - 1) / kAttnBM;
  e.mb_hi = mbs - 1;
  e.mb_count = mbs;
  e.n_splits = 1;
  e.split_keys = (q.n + c.key_tile - 1) / c.key_tile * c.key_tile;
  return e;
}

AttnEntry qdoc_entry(const Cfg &c, const Req &q, const Split &sp, int64_t part_row0,
                     const void *q_q, const void *k_cache, const void *v_cache, char *part_o,
                     float *part_lse) {
  AttnEntry e{};
  const size_t qrow = (size_t)c.hq * c.d * c.elem, krow = (size_t)c.hkv * c.d * c.elem;
  e.q = static_cast<const char *>(q_q) + q.q0 * qrow;
  e.k = static_cast<const char *>(k_cache) + q.tok0 * krow;
  e.v = static_cast<const char *>(v_cache) + q.tok0 * krow;
  e.o = nullptr;
  e.lse = nullptr;
  e.part_o = part_o + part_row0 * c.hq * c.d * c.elem;
  e.part_lse = part_lse + part_row0 * c.hq;
  e.n_rows = q.L_q;
  e.n_keys = q.L_d + q.L_q;
  const int mbs = qdoc_blocks(c, q.L_q);
  e.mb_hi = mbs - 1;
  e.mb_count = mbs;
  e.n_splits = sp.n_splits;
  e.split_keys = sp.split_keys;
  return e;
}

int entry_groups(const Cfg &c, const AttnEntry &e) { return e.mb_count * e.n_splits * c.hkv; }

daf_status_t run_entries(const Cfg &c, AttnKind kind, std::vector<AttnEntry> &entries, hipStream_t st) {
  for (size_t i0 = 0; i0 < entries.size(); i0 += kMaxEntries) {
    AttnLaunch p{};
    p.hq = c.hq;
    p.hkv = c.hkv;
    p.group = c.group;
    p.wgs_per_group = (kind == AttnKind::kQdoc && packed_qdoc(c)) ? 1 : c.group;
    p.scale_log2 = c.scale * 1.4426950408889634f;
    int groups = 0;
    const size_t i1 = std::min(entries.size(), i0 + kMaxEntries);
    for (size_t i = i0; i < i1; ++i) {
      AttnEntry e = entries[i];
      e.group0 = groups;
      groups += entry_groups(c, e);
      p.e[p.n_entries++] = e;
    }
    p.n_groups = groups;
    hipError_t err = launch_attention(c.dtype, c.d, kind, p, st);
    if (err != hipSuccess) return hip_fail(err, "attention launch");
  }
  return DAF_OK;
}

void add_self_entries(const Cfg &c, const Batch &b, const void *q_imp, const void *k_imp,
                      const void *v_imp, void *o_imp, float *lse_imp, std::vector<AttnEntry> &out,
                      void *hidden = nullptr, const int32_t *idx = nullptr) {
  // heaviest requests first: their top query blocks carry the most work
  std::vector<int> order;
  for (int i = 0; i < (int)b.r.size(); ++i)
    if (b.r[i].n > 0) order.push_back(i);
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) { return b.r[x].n > b.r[y].n; });
  for (int i : order) {
    AttnEntry e = self_entry(c, b.r[i], b.total_imp, q_imp, k_imp, v_imp, o_imp, lse_imp);
    if (hidden) {
      e.o2 = hidden;
      e.o2_idx = idx + b.r[i].imp0;
      e.o2_row0 = b.r[i].tok0;
    }
    out.push_back(e);
  }
}

// Stage-2 work of one call: the attention work table and the merge of the
// split partials.
struct QdocPlan {
  std::vector<AttnEntry> attn;
  std::vector<MergeEntry> merge;
};

daf_status_t qdoc_entries(const Cfg &c, const Batch &b, const void *q_q, const void *k_cache,
                          const void *v_cache, void *workspace, size_t ws_bytes, QdocPlan &plan, void *o_q,
                          float *lse_q, void *hidden = nullptr) {
  const std::vector<Split> sp = plan_splits(c, b);
  const WsLayout w = ws_layout(c, b, sp);
  if (w.part_rows == 0) return DAF_OK;
  if (!workspace) return fail(DAF_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", w.total);
  if (ws_bytes < w.total) return fail(DAF_ERR_WORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, w.total);
  if (reinterpret_cast<uintptr_t>(workspace) % 16 != 0)
    return fail(DAF_ERR_ALIGNMENT, "workspace is not 16-byte aligned");
  char *part_o = static_cast<char *>(workspace);
  float *part_lse = reinterpret_cast<float *>(static_cast<char *>(workspace) + w.part_o_bytes);
  int64_t prow = 0;
  const size_t qrow = (size_t)c.hq * c.d * c.elem;
  for (size_t i = 0; i < b.r.size(); ++i) {
    const Req &q = b.r[i];
    if (q.L_q == 0) continue;
    plan.attn.push_back(qdoc_entry(c, q, sp[i], prow, q_q, k_cache, v_cache, part_o, part_lse));
    MergeEntry m{};
    m.part_o = part_o + prow * c.hq * c.d * c.elem;
    m.part_lse = part_lse + prow * c.hq;
    m.o = static_cast<char *>(o_q) + q.q0 * qrow;
    m.lse = lse_q ? lse_q + q.q0 : nullptr;
    m.lse_stride = (int32_t)b.total_q;
    m.n_rows = q.L_q;
    m.n_splits = sp[i].n_splits;
    if (hidden) {
      m.o2 = hidden;
      m.o2_row0 = q.tok0 + q.L_d;
    }
    plan.merge.push_back(m);
    prow += (int64_t)q.L_q * sp[i].n_splits;
  }
  return DAF_OK;
}

daf_status_t run_merge(const Cfg &c, std::vector<MergeEntry> &merge, hipStream_t st) {
  for (size_t i0 = 0; i0 < merge.size(); i0 += kMaxEntries) {
    MergeLaunch p{};
    p.hq = c.hq;
    int rows = 0;
    const size_t i1 = std::min(merge.size(), i0 + kMaxEntries);
    for (size_t i = i0; i < i1; ++i) {
      MergeEntry m = merge[i];
      m.row0 = rows;
      rows += m.n_rows;
      p.e[p.n_entries++] = m;
    }
    p.total_rows = rows;
    hipError_t err = c.dtype == DAF_BF16 ? launch_qdoc_merge_bf16(c.d, p, st) : launch_merge(c.dtype, c.d, p, st);
    if (err != hipSuccess) return hip_fail(err, "merge launch");
  }
  return DAF_OK;
}

// Stage 2 and its merge.
daf_status_t run_qdoc(const Cfg &c, QdocPlan &plan, hipStream_t st) {
  CHECK(run_entries(c, AttnKind::kQdoc, plan.attn, st));
  return run_merge(c, plan.merge, st);
}

// ---- row movement ---------------------------------------------------------------
template <typename F>
daf_status_t for_row_groups(const Batch &b, const int32_t *idx, int64_t row_bytes, int layout_docs,
                            F &&fn) {
  const int nreq = (int)b.r.size();
  for (int i0 = 0; i0 < nreq; i0 += kMaxRowReqs) {
    RowLaunch p{};
    p.units = (int32_t)(row_bytes / 16);
    p.idx = idx;
    const int i1 = std::min(nreq, i0 + kMaxRowReqs);
    int64_t cu_doc = 0;
    for (int i = 0; i < i0; ++i) cu_doc += b.r[i].L_d;
    for (int i = i0; i < i1; ++i) {
      const Req &q = b.r[i];
      RowReq &r = p.r[p.n_req++];
      r.base = layout_docs ? cu_doc : q.tok0;
      r.imp0 = q.imp0;
      r.n_imp = q.n;
      r.q0 = q.q0;
      r.n_q = q.L_q;
      r.L_d = q.L_d;
      p.total_imp += q.n;
      p.total_q += q.L_q;
      cu_doc += q.L_d;
    }
    CHECK(fn(p));
  }
  return DAF_OK;
}

daf_status_t fuse_impl(const Cfg &c, const Batch &b, uint32_t flags, const int32_t *idx,
                       const void *k_imp, const void *v_imp, const void *k_q, const void *v_q,
                       void *k_cache, void *v_cache, const void *o_imp, const void *o_q, void *hidden,
                       hipStream_t st) {
  if (flags & DAF_FUSE_KV) {
    ScatterPair pr[2] = {{k_imp, k_q, k_cache}, {v_imp, v_q, v_cache}};
    CHECK(for_row_groups(b, idx, (int64_t)c.hkv * c.d * c.elem, 0, [&](const RowLaunch &p) {
      hipError_t e = launch_scatter(p, pr, 2, st);
      return e == hipSuccess ? DAF_OK : hip_fail(e, "KV fuse launch");
    }));
  }
  if (flags & DAF_FUSE_HIDDEN) {
    ScatterPair pr[1] = {{o_imp, o_q, hidden}};
    CHECK(for_row_groups(b, idx, (int64_t)c.hq * c.d * c.elem, 0, [&](const RowLaunch &p) {
      hipError_t e = launch_scatter(p, pr, 1, st);
      return e == hipSuccess ? DAF_OK : hip_fail(e, "hidden fuse launch");
    }));
  }
  return DAF_OK;
}

daf_status_t check_fuse_ptrs(const Batch &b, uint32_t flags, const int32_t *idx, const void *k_imp,
                             const void *v_imp, const void *k_q, const void *v_q, void *k_cache,
                             void *v_cache, const void *o_imp, const void *o_q, void *hidden) {
  if ((flags & ~(uint32_t)(DAF_FUSE_KV | DAF_FUSE_HIDDEN)) != 0 || flags == 0)
    return fail(DAF_ERR_INVALID_ARG, "flags=%u (use DAF_FUSE_KV and/or DAF_FUSE_HIDDEN)", flags);
  const bool imp = b.total_imp > 0, qs = b.total_q > 0;
  if (imp) CHECK(need_ptr(idx, "idx"));
  if (flags & DAF_FUSE_KV) {
    if (imp) {
      CHECK(need_ptr(k_imp, "k_imp"));
      CHECK(need_ptr(v_imp, "v_imp"));
    }
    if (qs) {
      CHECK(need_ptr(k_q, "k_q"));
      CHECK(need_ptr(v_q, "v_q"));
    }
    if (imp || qs) {
      CHECK(need_ptr(k_cache, "k_cache"));
      CHECK(need_ptr(v_cache, "v_cache"));
    }
  }
  if (flags & DAF_FUSE_HIDDEN) {
    if (imp) CHECK(need_ptr(o_imp, "o_imp"));
    if (qs) CHECK(need_ptr(o_q, "o_q"));
    if (imp || qs) CHECK(need_ptr(hidden, "hidden"));
  }
  return DAF_OK;
}

// The layer's attention: hybrid KV write-back, stage 2 with its merge, and
// stage 1 (on the second stream); with `hidden` set, the stage epilogues also
// fuse the outputs into it. Pointers are checked by the caller.
daf_status_t layer_attn_impl(const Cfg &c, const Batch &b, const int32_t *idx, const void *q_imp,
                             const void *k_imp, const void *v_imp, const void *q_q, const void *k_q,
                             const void *v_q, void *k_cache, void *v_cache, void *o_imp, float *lse_imp, void *o_q,
                             float *lse_q, void *hidden, void *workspace, size_t ws_bytes, hipStream_t stream,
                             bool fork = true) {
  // plan (and check the workspace) before enqueueing anything
  std::vector<AttnEntry> self;
  QdocPlan qdoc;
  // the epilogues also fuse the outputs into the hidden states: stage-1 row i
  // of request b goes to hidden[tok_b + idx[i]], question row j (written by
  // the merge) to hidden[tok_b + L_d,b + j]
  add_self_entries(c, b, q_imp, k_imp, v_imp, o_imp, lse_imp, self, hidden, idx);
  CHECK(qdoc_entries(c, b, q_q, k_cache, v_cache, workspace, ws_bytes, qdoc, o_q, lse_q, hidden));
  // Stage 1 reads only the condensed q/k/v and writes o_imp and the
  // important rows of hidden; the hybrid KV (which stage 2 reads), stage 2
  // and the merge (question rows of hidden) touch none of that, so stage 1
  // runs beside them on the second stream.
  std::lock_guard<std::mutex> lock(g_aux_mu);
  AuxStream *ax = (self.empty() || !fork) ? nullptr : aux_stream();
  daf_status_t st1 = DAF_OK;
  daf_status_t st = fuse_impl(c, b, DAF_FUSE_KV, idx, k_imp, v_imp, k_q, v_q, k_cache, v_cache, nullptr,
                              nullptr, nullptr, stream);
  // the fork point follows the KV write-back, and stage 2 and the merge are
  // enqueued before stage 1, so stage 2's workgroups are dispatched first and
  // stage 1 fills in behind them (measured 1-2% faster than stage 1 first)
  hipError_t ef = ax ? hipEventRecord(ax->fork, stream) : hipSuccess;
  if (st == DAF_OK) st = run_qdoc(c, qdoc, stream);
  if (ax) {
    if (ef == hipSuccess) ef = hipStreamWaitEvent(ax->s, ax->fork, 0);
    if (ef != hipSuccess) return hip_fail(ef, "stream fork");
    st1 = run_entries(c, AttnKind::kSelf, self, ax->s);
    // always join, so that nothing the caller's stream runs next can race stage 1
    hipError_t e = hipEventRecord(ax->join, ax->s);
    if (e == hipSuccess) e = hipStreamWaitEvent(stream, ax->join, 0);
    if (e != hipSuccess) return hip_fail(e, "stream join");
  } else if (st == DAF_OK) {
    st = run_entries(c, AttnKind::kSelf, self, stream);
  }
  CHECK(st1);
  CHECK(st);
  return ok();
}

// ---- decoder layer around the attention -------------------------------------
struct LayerWs {
  int64_t rows;
  size_t h, q, k, v, o, m, attn, attn_bytes, part, total;  // byte offsets, total size
};

daf_status_t check_weights(const Cfg &c, const daf_layer_weights_t *w) {
  if (!w) return fail(DAF_ERR_INVALID_ARG, "weights is NULL");
  if (c.dtype != DAF_BF16) return fail(DAF_ERR_UNSUPPORTED, "the decoder layer runs in bf16 only");
  if (w->hidden <= 0 || w->hidden % 128 != 0 || w->inter <= 0 || w->inter % 128 != 0)
    return fail(DAF_ERR_UNSUPPORTED, "hidden=%d and inter=%d must be positive multiples of 128", w->hidden,
                w->inter);
  if (((int64_t)w->inter + 256) * w->hidden * 2 > INT32_MAX || (int64_t)w->hidden * w->inter * 2 > INT32_MAX)
    return fail(DAF_ERR_UNSUPPORTED, "hidden=%d x inter=%d too large", w->hidden, w->inter);
  if ((c.hq * c.d) % 128 != 0 || (c.hkv * c.d) % 128 != 0)
    return fail(DAF_ERR_UNSUPPORTED, "Hq*D=%d and Hkv*D=%d must be multiples of 128", c.hq * c.d, c.hkv * c.d);
  if (!(w->eps >= 0.f) || !(w->rope_theta > 0.f))
    return fail(DAF_ERR_INVALID_ARG, "eps must be >= 0 and rope_theta > 0");
  const void *p[] = {w->w_in, w->wq, w->bq, w->wk, w->bk, w->wv, w->bv, w->wo, w->w_post, w->wgu, w->wd};
  const char *n[] = {"w_in", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "w_post", "wgu", "wd"};
  for (int i = 0; i < 11; ++i) CHECK(need_ptr(p[i], n[i]));
  return DAF_OK;
}

LayerWs layer_ws(const Cfg &c, const daf_layer_weights_t &w, const Batch &b, int mode) {
  LayerWs l{};
  l.rows = mode == DAF_LAYER_DAF ? b.total_imp + b.total_q : b.total_tok;
  const size_t r = (size_t)l.rows, e = 2;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
  };
  l.h = take(r * w.hidden * e);
  l.q = take(r * c.hq * c.d * e);
  l.k = take(r * c.hkv * c.d * e);
  l.v = take(r * c.hkv * c.d * e);
  l.o = take(r * c.hq * c.d * e);
  l.m = take(r * w.inter * e);
  l.attn_bytes = mode == DAF_LAYER_DAF ? ws_layout(c, b, plan_splits(c, b)).total : 0;
  l.attn = take(l.attn_bytes);
  l.part = take(kGemmPartBytes);  // fp32 k pieces of the projections' tail tiles
  l.total = off;
  return l;
}

// part: workspace for the k pieces of tail tiles (kGemmPartBytes), or null
daf_status_t gemm(int64_t M, int N, int K, const void *A, const void *W, const void *bias, const void *res, void *C,
                  hipStream_t st, float *part = nullptr) {
  GemmArgs g{};
  g.A = A;
  g.W = W;
  g.bias = bias;
  g.residual = res;
  g.C = C;
  g.M = M;
  g.N = N;
  g.K = K;
  const hipError_t e = part ? launch_gemm_split(g, part, kGemmPartBytes, st) : launch_gemm(g, st);
  return e == hipSuccess ? DAF_OK : hip_fail(e, "linear launch");
}

}  // namespace

extern "C" {

const char *daf_status_string(daf_status_t s) {
  switch (s) {
    case DAF_OK: return "DAF_OK";
    case DAF_ERR_INVALID_ARG: return "DAF_ERR_INVALID_ARG";
    case DAF_ERR_ALIGNMENT: return "DAF_ERR_ALIGNMENT";
    case DAF_ERR_UNSUPPORTED: return "DAF_ERR_UNSUPPORTED";
    case DAF_ERR_WORKSPACE: return "DAF_ERR_WORKSPACE";
    case DAF_ERR_HIP: return "DAF_ERR_HIP";
  }
  return "DAF_ERR_UNKNOWN";
}

const char *daf_last_error(void) { return g_err; }

int32_t daf_version(void) { return 100; }

daf_status_t daf_gather_important(const daf_batch_t *batch, int32_t src_layout, const void *src,
                                  int64_t row_bytes, const int32_t *idx, void *dst,
                                  hipStream_t stream) {
  try {
    Batch b;
    CHECK(parse_batch(batch, b));
    if (src_layout != DAF_SRC_TOKENS && src_layout != DAF_SRC_DOCS)
      return fail(DAF_ERR_INVALID_ARG, "src_layout=%d", src_layout);
    if (row_bytes <= 0) return fail(DAF_ERR_INVALID_ARG, "row_bytes=%lld must be > 0", (long long)row_bytes);
    if (row_bytes % 16 != 0) return fail(DAF_ERR_ALIGNMENT, "row_bytes=%lld is not a multiple of 16", (long long)row_bytes);
    if (row_bytes / 16 > INT32_MAX) return fail(DAF_ERR_UNSUPPORTED, "row_bytes too large");
    if (b.total_imp == 0) return ok();
    CHECK(need_ptr(src, "src"));
    CHECK(need_ptr(idx, "idx"));
    CHECK(need_ptr(dst, "dst"));
    CHECK(for_row_groups(b, idx, row_bytes, src_layout == DAF_SRC_DOCS, [&](const RowLaunch &p) {
      hipError_t e = launch_gather(p, 0, src, dst, stream);
      return e == hipSuccess ? DAF_OK : hip_fail(e, "gather launch");
    }));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_imp_self_attn(const daf_attn_cfg_t *cfg, const daf_batch_t *batch, const void *q_imp,
                               const void *k_imp, const void *v_imp, void *o_imp, float *lse_imp,
                               hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    CHECK(check_kv_extent(c, b));
    if (b.total_imp == 0) return ok();
    CHECK(need_ptr(q_imp, "q_imp"));
    CHECK(need_ptr(k_imp, "k_imp"));
    CHECK(need_ptr(v_imp, "v_imp"));
    CHECK(need_ptr(o_imp, "o_imp"));
    if (lse_imp) CHECK(need_ptr(lse_imp, "lse_imp"));
    std::vector<AttnEntry> entries;
    add_self_entries(c, b, q_imp, k_imp, v_imp, o_imp, lse_imp, entries);
    CHECK(run_entries(c, AttnKind::kSelf, entries, stream));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_position_attn(const daf_attn_cfg_t *cfg, int32_t n_rows, int32_t n_keys, const void *q,
                               const int32_t *q_pos, const void *k, const void *v, void *o, float *lse,
                               hipStream_t stream) {
  try {
    Cfg c;
    CHECK(parse_cfg(cfg, c));
    if (n_rows < 0 || n_keys < 0) return fail(DAF_ERR_INVALID_ARG, "n_rows=%d, n_keys=%d must be >= 0", n_rows, n_keys);
    if (!q_pos && n_rows > n_keys)
      return fail(DAF_ERR_INVALID_ARG, "without q_pos, n_rows=%d must not exceed n_keys=%d", n_rows, n_keys);
    if (q_pos && n_rows > 0 && n_keys == 0) return fail(DAF_ERR_INVALID_ARG, "n_keys is 0 but rows have positions");
    if ((int64_t)n_keys * c.hkv * c.d * c.elem > INT32_MAX)
      return fail(DAF_ERR_UNSUPPORTED, "%lld K/V bytes exceed 2 GiB", (long long)n_keys * c.hkv * c.d * c.elem);
    if (n_rows == 0) return ok();
    CHECK(need_ptr(q, "q"));
    CHECK(need_ptr(k, "k"));
    CHECK(need_ptr(v, "v"));
    CHECK(need_ptr(o, "o"));
    if (lse) CHECK(need_ptr(lse, "lse"));
    if (q_pos && reinterpret_cast<uintptr_t>(q_pos) % 4 != 0) return fail(DAF_ERR_ALIGNMENT, "q_pos is not 4-byte aligned");
    AttnEntry e{};
    e.q = q;
    e.k = k;
    e.v = v;
    e.o = o;
    e.lse = lse;
    e.lse_stride = n_rows;
    e.n_rows = n_rows;
    e.n_keys = n_keys;
    const int mbs = (n_rows + kAttnBM - 1) / kAttnBM;
    e.mb_hi = mbs - 1;
    e.mb_count = mbs;
    e.n_splits = 1;
    e.split_keys = (n_keys + c.key_tile - 1) / c.key_tile * c.key_tile;
    e.q_pos = q_pos;
    std::vector<AttnEntry> entries{e};
    CHECK(run_entries(c, AttnKind::kSelf, entries, stream));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_select_important(const daf_attn_cfg_t *cfg, const daf_batch_t *batch, int32_t n_layers,
                                  const void *const *k_fresh, const void *const *k_cached, float *scores,
                                  int32_t *idx, hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    if (n_layers < 1 || n_layers > kMaxSelectLayers)
      return fail(DAF_ERR_INVALID_ARG, "n_layers=%d (supported: 1..%d)", n_layers, kMaxSelectLayers);
    const int64_t row_bytes = (int64_t)c.hkv * c.d * c.elem;
    if (row_bytes > 4096)
      return fail(DAF_ERR_UNSUPPORTED, "Hkv*D*element = %lld bytes per token exceeds 4096", (long long)row_bytes);
    const int64_t rows = b.total_tok - b.total_q;  // document rows
    if (rows == 0) return ok();
    if (!k_fresh || !k_cached) return fail(DAF_ERR_INVALID_ARG, "k_fresh and k_cached must be non-NULL host arrays");
    SelectLaunch p{};
    for (int l = 0; l < n_layers; ++l) {
      CHECK(need_ptr(k_fresh[l], "k_fresh[l]"));
      CHECK(need_ptr(k_cached[l], "k_cached[l]"));
      p.fresh[l] = k_fresh[l];
      p.cached[l] = k_cached[l];
    }
    CHECK(need_ptr(scores, "scores"));
    if (b.total_imp > 0) CHECK(need_ptr(idx, "idx"));
    p.scores = scores;
    p.idx = idx;
    p.rows = rows;
    p.row_bytes = (int32_t)row_bytes;
    p.n_layers = n_layers;
    hipError_t e = launch_select_scores(p, c.dtype == DAF_BF16, stream);
    if (e != hipSuccess) return hip_fail(e, "selection score launch");
    int64_t doc0 = 0;
    for (size_t i = 0; i < b.r.size(); ++i) {
      const Req &q = b.r[i];
      if (q.n > 0) {
        p.req[p.n_req++] = SelectReq{doc0, q.L_d, q.n, q.imp0};
        if (p.n_req == kMaxSelectReqs) {
          e = launch_select_topn(p, stream);
          if (e != hipSuccess) return hip_fail(e, "selection launch");
          p.n_req = 0;
        }
      }
      doc0 += q.L_d;
    }
    e = launch_select_topn(p, stream);
    if (e != hipSuccess) return hip_fail(e, "selection launch");
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_linear(int64_t M, int32_t N, int32_t K, const void *A, const void *W, const void *bias,
                        const void *residual, void *C, hipStream_t stream) {
  try {
    if (M < 0) return fail(DAF_ERR_INVALID_ARG, "M=%lld is negative", (long long)M);
    if (N <= 0 || N % 128 != 0) return fail(DAF_ERR_UNSUPPORTED, "N=%d is not a positive multiple of 128", N);
    if (K <= 0 || K % 64 != 0) return fail(DAF_ERR_UNSUPPORTED, "K=%d is not a positive multiple of 64", K);
    if ((int64_t)K * 2 * 128 > INT32_MAX) return fail(DAF_ERR_UNSUPPORTED, "K=%d too large", K);
    if (M == 0) return ok();
    CHECK(need_ptr(A, "A"));
    CHECK(need_ptr(W, "W"));
    CHECK(need_ptr(C, "C"));
    if (bias) CHECK(need_ptr(bias, "bias"));
    if (residual) CHECK(need_ptr(residual, "residual"));
    GemmArgs g{};
    g.A = A;
    g.W = W;
    g.bias = bias;
    g.residual = residual;
    g.C = C;
    g.M = M;
    g.N = N;
    g.K = K;
    const hipError_t e = launch_gemm(g, stream);
    if (e != hipSuccess) return hip_fail(e, "linear launch");
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_linear_swiglu(int64_t M, int32_t I, int32_t K, const void *A, const void *Wgu, void *C,
                               hipStream_t stream) {
  try {
    if (M < 0) return fail(DAF_ERR_INVALID_ARG, "M=%lld is negative", (long long)M);
    if (I <= 0 || I % 64 != 0) return fail(DAF_ERR_UNSUPPORTED, "I=%d is not a positive multiple of 64", I);
    if (K <= 0 || K % 64 != 0) return fail(DAF_ERR_UNSUPPORTED, "K=%d is not a positive multiple of 64", K);
    if (((int64_t)I + 256) * K * 2 > INT32_MAX) return fail(DAF_ERR_UNSUPPORTED, "I*K too large");
    if (M == 0) return ok();
    CHECK(need_ptr(A, "A"));
    CHECK(need_ptr(Wgu, "Wgu"));
    CHECK(need_ptr(C, "C"));
    GemmArgs g{};
    g.A = A;
    g.W = Wgu;
    g.C = C;
    g.M = M;
    g.N = I;
    g.K = K;
    g.glu = 1;
    const hipError_t e = launch_gemm(g, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "linear launch");
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_rmsnorm(int64_t rows, int32_t width, const void *x, const void *w, float eps, void *y,
                         hipStream_t stream) {
  try {
    if (rows < 0) return fail(DAF_ERR_INVALID_ARG, "rows=%lld is negative", (long long)rows);
    if (width <= 0 || width % 8 != 0) return fail(DAF_ERR_UNSUPPORTED, "width=%d is not a positive multiple of 8", width);
    if (!(eps >= 0.f)) return fail(DAF_ERR_INVALID_ARG, "eps must be >= 0");
    if (rows == 0) return ok();
    CHECK(need_ptr(x, "x"));
    CHECK(need_ptr(w, "w"));
    CHECK(need_ptr(y, "y"));
    const hipError_t e = launch_rmsnorm(rows, width, x, w, eps, y, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "rmsnorm launch");
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_rope(int64_t rows, int32_t n_heads, int32_t head_dim, int64_t row_stride, void *x,
                      const int32_t *pos, float theta, hipStream_t stream) {
  try {
    if (rows < 0) return fail(DAF_ERR_INVALID_ARG, "rows=%lld is negative", (long long)rows);
    if (n_heads <= 0 || head_dim <= 0 || head_dim % 2 != 0)
      return fail(DAF_ERR_INVALID_ARG, "n_heads=%d, head_dim=%d (head_dim must be even)", n_heads, head_dim);
    if (row_stride < (int64_t)n_heads * head_dim)
      return fail(DAF_ERR_INVALID_ARG, "row_stride=%lld is below n_heads * head_dim", (long long)row_stride);
    if (!(theta > 0.f)) return fail(DAF_ERR_INVALID_ARG, "theta must be > 0");
    if (rows == 0) return ok();
    if (!x || !pos) return fail(DAF_ERR_INVALID_ARG, "x and pos must be non-NULL");
    if (reinterpret_cast<uintptr_t>(x) % 2 != 0 || reinterpret_cast<uintptr_t>(pos) % 4 != 0)
      return fail(DAF_ERR_ALIGNMENT, "x must be 2-byte and pos 4-byte aligned");
    const hipError_t e = launch_rope(rows, n_heads, head_dim, row_stride, x, pos, theta, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "rope launch");
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_silu_mul(int64_t rows, int32_t width, const void *gu, void *out, hipStream_t stream) {
  try {
    if (rows < 0) return fail(DAF_ERR_INVALID_ARG, "rows=%lld is negative", (long long)rows);
    if (width <= 0 || width % 8 != 0) return fail(DAF_ERR_UNSUPPORTED, "width=%d is not a positive multiple of 8", width);
    if (rows == 0) return ok();
    CHECK(need_ptr(gu, "gu"));
    CHECK(need_ptr(out, "out"));
    const hipError_t e = launch_silu_mul(rows, width, gu, out, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "silu_mul launch");
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

size_t daf_decoder_layer_workspace_size(const daf_attn_cfg_t *cfg, const daf_layer_weights_t *w,
                                        const daf_batch_t *batch, int32_t mode) {
  try {
    Cfg c;
    Batch b;
    if (parse_cfg(cfg, c) != DAF_OK || parse_batch(batch, b) != DAF_OK || !w) return 0;
    if (mode != DAF_LAYER_DAF && mode != DAF_LAYER_FULL) return 0;
    return layer_ws(c, *w, b, mode).total;
  } catch (...) {
    return 0;
  }
}

daf_status_t daf_decoder_layer(const daf_attn_cfg_t *cfg, const daf_layer_weights_t *w, const daf_batch_t *batch,
                               int32_t mode, const int32_t *idx, const int32_t *pos, void *x, void *k_cache,
                               void *v_cache, void *workspace, size_t ws_bytes, hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    CHECK(check_weights(c, w));
    if (mode != DAF_LAYER_DAF && mode != DAF_LAYER_FULL)
      return fail(DAF_ERR_INVALID_ARG, "mode=%d (use DAF_LAYER_DAF or DAF_LAYER_FULL)", mode);
    CHECK(check_kv_extent(c, b));
    const LayerWs l = layer_ws(c, *w, b, mode);
    if (l.rows == 0) return ok();
    CHECK(need_ptr(x, "x"));
    if (!pos || reinterpret_cast<uintptr_t>(pos) % 4 != 0)
      return fail(DAF_ERR_INVALID_ARG, "pos must be a non-NULL, 4-byte aligned int32 array");
    if (mode == DAF_LAYER_DAF) {
      if (b.total_imp > 0) CHECK(need_ptr(idx, "idx"));
      CHECK(need_ptr(k_cache, "k_cache"));
      CHECK(need_ptr(v_cache, "v_cache"));
    }
    if (!workspace) return fail(DAF_ERR_WORKSPACE, "workspace is NULL (need %zu bytes)", l.total);
    if (ws_bytes < l.total) return fail(DAF_ERR_WORKSPACE, "workspace has %zu bytes, need %zu", ws_bytes, l.total);
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
      return fail(DAF_ERR_ALIGNMENT, "workspace is not %zu-byte aligned", kAlign);
    char *ws = static_cast<char *>(workspace);
    void *h = ws + l.h, *q = ws + l.q, *k = ws + l.k, *v = ws + l.v, *o = ws + l.o, *m = ws + l.m;
    const int64_t R = l.rows;
    const int H = w->hidden, I = w->inter, QW = c.hq * c.d, KW = c.hkv * c.d;
    const hipError_t e0 = launch_rmsnorm(R, H, x, w->w_in, w->eps, h, stream);
    if (e0 != hipSuccess) return hip_fail(e0, "rmsnorm launch");
    float *part = reinterpret_cast<float *>(ws + l.part);
    CHECK(gemm(R, QW, H, h, w->wq, w->bq, nullptr, q, stream, part));
    CHECK(gemm(R, KW, H, h, w->wk, w->bk, nullptr, k, stream, part));
    CHECK(gemm(R, KW, H, h, w->wv, w->bv, nullptr, v, stream, part));
    hipError_t e1 = launch_rope(R, c.hq, c.d, QW, q, pos, w->rope_theta, stream);
    if (e1 == hipSuccess) e1 = launch_rope(R, c.hkv, c.d, KW, k, pos, w->rope_theta, stream);
    if (e1 != hipSuccess) return hip_fail(e1, "rope launch");
    if (mode == DAF_LAYER_DAF) {
      const int64_t ni = b.total_imp;
      char *qb = static_cast<char *>(q), *kb = static_cast<char *>(k), *vb = static_cast<char *>(v);
      char *ob = static_cast<char *>(o);
      CHECK(layer_attn_impl(c, b, idx, qb, kb, vb, qb + ni * QW * 2, kb + ni * KW * 2, vb + ni * KW * 2, k_cache,
                            v_cache, ob, nullptr, ob + ni * QW * 2, nullptr, nullptr, ws + l.attn, l.attn_bytes,
                            stream));
    } else {
      // every token recomputed: causal attention over each request's own rows
      std::vector<int> order;
      for (int i = 0; i < (int)b.r.size(); ++i)
        if (b.r[i].L_d + b.r[i].L_q > 0) order.push_back(i);
      std::stable_sort(order.begin(), order.end(), [&](int a, int bb) {
        return b.r[a].L_d + b.r[a].L_q > b.r[bb].L_d + b.r[bb].L_q;
      });
      std::vector<AttnEntry> entries;
      for (int i : order) {
        const Req &r = b.r[i];
        const int T = r.L_d + r.L_q;
        AttnEntry e{};
        e.q = static_cast<char *>(q) + r.tok0 * QW * 2;
        e.k = static_cast<char *>(k) + r.tok0 * KW * 2;
        e.v = static_cast<char *>(v) + r.tok0 * KW * 2;
        e.o = static_cast<char *>(o) + r.tok0 * QW * 2;
        e.n_rows = T;
        e.n_keys = T;
        const int mbs = (T + kAttnBM - 1) / kAttnBM;
        e.mb_hi = mbs - 1;
        e.mb_count = mbs;
        e.n_splits = 1;
        e.split_keys = (T + c.key_tile - 1) / c.key_tile * c.key_tile;
        entries.push_back(e);
      }
      CHECK(run_entries(c, AttnKind::kSelf, entries, stream));
    }
    CHECK(gemm(R, H, QW, o, w->wo, nullptr, x, x, stream, part));
    const hipError_t e2 = launch_rmsnorm(R, H, x, w->w_post, w->eps, h, stream);
    if (e2 != hipSuccess) return hip_fail(e2, "rmsnorm launch");
    {  // gate and up projections with SiLU(gate) * up in the epilogue
      GemmArgs g{};
      g.A = h;
      g.W = w->wgu;
      g.C = m;
      g.M = R;
      g.N = I;
      g.K = H;
      g.glu = 1;
      const hipError_t e3 = launch_gemm(g, stream);
      if (e3 != hipSuccess) return hip_fail(e3, "linear launch");
    }
    CHECK(gemm(R, H, I, m, w->wd, nullptr, x, x, stream, part));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

size_t daf_qdoc_workspace_size(const daf_attn_cfg_t *cfg, const daf_batch_t *batch) {
  try {
    Cfg c;
    Batch b;
    if (parse_cfg(cfg, c) != DAF_OK || parse_batch(batch, b) != DAF_OK) return 0;
    const WsLayout w = ws_layout(c, b, plan_splits(c, b));
    return w.part_rows ? w.total : 0;
  } catch (...) {
    return 0;
  }
}

size_t daf_layer_workspace_size(const daf_attn_cfg_t *cfg, const daf_batch_t *batch) {
  return daf_qdoc_workspace_size(cfg, batch);
}

daf_status_t daf_qdoc_attn(const daf_attn_cfg_t *cfg, const daf_batch_t *batch, const void *q_q,
                           const void *k_cache, const void *v_cache, void *o_q, float *lse_q,
                           void *workspace, size_t ws_bytes, hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    CHECK(check_kv_extent(c, b));
    if (b.total_q == 0) return ok();
    CHECK(need_ptr(q_q, "q_q"));
    CHECK(need_ptr(k_cache, "k_cache"));
    CHECK(need_ptr(v_cache, "v_cache"));
    CHECK(need_ptr(o_q, "o_q"));
    if (lse_q) CHECK(need_ptr(lse_q, "lse_q"));
    QdocPlan plan;
    CHECK(qdoc_entries(c, b, q_q, k_cache, v_cache, workspace, ws_bytes, plan, o_q, lse_q));
    CHECK(run_qdoc(c, plan, stream));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_fuse(const daf_attn_cfg_t *cfg, const daf_batch_t *batch, uint32_t flags,
                      const int32_t *idx, const void *k_imp, const void *v_imp, const void *k_q,
                      const void *v_q, void *k_cache, void *v_cache, const void *o_imp,
                      const void *o_q, void *hidden, hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    CHECK(check_fuse_ptrs(b, flags, idx, k_imp, v_imp, k_q, v_q, k_cache, v_cache, o_imp, o_q, hidden));
    CHECK(fuse_impl(c, b, flags, idx, k_imp, v_imp, k_q, v_q, k_cache, v_cache, o_imp, o_q, hidden, stream));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_layer_attn(const daf_attn_cfg_t *cfg, const daf_batch_t *batch, const int32_t *idx,
                            const void *q_imp, const void *k_imp, const void *v_imp, const void *q_q,
                            const void *k_q, const void *v_q, void *k_cache, void *v_cache,
                            void *o_imp, float *lse_imp, void *o_q, float *lse_q, void *hidden,
                            void *workspace, size_t ws_bytes, hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    CHECK(check_kv_extent(c, b));
    const uint32_t both = DAF_FUSE_KV | DAF_FUSE_HIDDEN;
    if (b.total_imp == 0 && b.total_q == 0) return ok();
    CHECK(check_fuse_ptrs(b, both, idx, k_imp, v_imp, k_q, v_q, k_cache, v_cache, o_imp, o_q, hidden));
    if (b.total_imp > 0) CHECK(need_ptr(q_imp, "q_imp"));
    if (b.total_q > 0) CHECK(need_ptr(q_q, "q_q"));
    if (lse_imp) CHECK(need_ptr(lse_imp, "lse_imp"));
    if (lse_q) CHECK(need_ptr(lse_q, "lse_q"));
    return layer_attn_impl(c, b, idx, q_imp, k_imp, v_imp, q_q, k_q, v_q, k_cache, v_cache, o_imp, lse_imp, o_q,
                           lse_q, hidden, workspace, ws_bytes, stream);
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

size_t daf_layer_noalloc_max_bytes(void) { return kScratchBytes; }

daf_status_t daf_layer_attn_noalloc(const daf_attn_cfg_t *cfg, const daf_batch_t *batch, const int32_t *idx,
                                    const void *q_imp, const void *k_imp, const void *v_imp, const void *q_q,
                                    const void *k_q, const void *v_q, void *k_cache, void *v_cache, void *o_imp,
                                    float *lse_imp, void *o_q, float *lse_q, void *hidden, hipStream_t stream) {
  try {
    Cfg c;
    Batch b;
    CHECK(parse_cfg(cfg, c));
    CHECK(parse_batch(batch, b));
    CHECK(check_kv_extent(c, b));
    const uint32_t both = DAF_FUSE_KV | DAF_FUSE_HIDDEN;
    if (b.total_imp == 0 && b.total_q == 0) return ok();
    CHECK(check_fuse_ptrs(b, both, idx, k_imp, v_imp, k_q, v_q, k_cache, v_cache, o_imp, o_q, hidden));
    if (b.total_imp > 0) CHECK(need_ptr(q_imp, "q_imp"));
    if (b.total_q > 0) CHECK(need_ptr(q_q, "q_q"));
    if (lse_imp) CHECK(need_ptr(lse_imp, "lse_imp"));
    if (lse_q) CHECK(need_ptr(lse_q, "lse_q"));
    const size_t need = ws_layout(c, b, plan_splits(c, b)).total;
    if (need > kScratchBytes)
      return fail(DAF_ERR_WORKSPACE, "this batch needs %zu bytes of scratch; the allocation-free call has %zu",
                  need, kScratchBytes);
    hipError_t e = hipSuccess;
    void *ws = scratch_ptr(e);
    if (!ws) return hip_fail(e, "scratch address lookup");
    // one stream: the second stream of daf_layer_attn is created on first use
    return layer_attn_impl(c, b, idx, q_imp, k_imp, v_imp, q_q, k_q, v_q, k_cache, v_cache, o_imp, lse_imp, o_q,
                           lse_q, hidden, ws, kScratchBytes, stream, false);
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

daf_status_t daf_check_indices(const daf_batch_t *batch, const int32_t *idx, int32_t *d_bad_count,
                               hipStream_t stream) {
  try {
    Batch b;
    CHECK(parse_batch(batch, b));
    CHECK(need_ptr(d_bad_count, "d_bad_count"));
    if (b.total_imp > 0) CHECK(need_ptr(idx, "idx"));
    int first = 1;
    CHECK(for_row_groups(b, idx, 16, 0, [&](const RowLaunch &p) {
      hipError_t e = launch_check_indices(p, d_bad_count, first ? 0 : 1, stream);
      first = 0;
      return e == hipSuccess ? DAF_OK : hip_fail(e, "check launch");
    }));
    return ok();
  } catch (...) {
    return fail(DAF_ERR_HIP, "unexpected host exception");
  }
}

}  // extern "C"
