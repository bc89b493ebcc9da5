"""DAF CPU oracle: the plain definition of the per-layer DAF attention.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package. It shares no code with
the HIP product library and the product never calls it.

The arithmetic lives in ``daf_oracle.c`` (fp64 accumulation, explicit masks,
three-pass softmax). This module loads it with ctypes and composes the layer in
the order the paper gives (Sec. 2):

  1. hybrid KV cache: the important tokens' recomputed K/V replace the offline
     rows before question-document attention (Sec. 2 item 2), and the
     question's own K/V follow the documents (the question's keys are every
     document token and the question's own tokens);
  2. stage 1, important-token self-attention over the condensed sequence
     (Sec. 2 item 1; important tokens see only each other, Complexity
     Analysis);
  3. stage 2, question rows over all L_d + L_q keys (Sec. 2 item 2);
  4. state fusion: stage outputs written into the hidden-state rows of their
     tokens (Sec. 2 item 3).

The step before the path, important-token selection (Sec. 2 item 1), is given
as a score per document token (KV deviation averaged over the selection
layers) and a top-n choice returned in original order. For the comparison with
the schemes the Complexity Analysis contrasts DAF with, it also gives full recomputation (causal attention over every token) and
the CacheBlend pattern (important and question tokens over the full context,
causal by original position).

Arrays are numpy. Raw buffers (bf16 bit patterns as uint16, or float32) are
moved byte for byte; attention inputs are float32 and outputs are float64.
Parity is pinned by the CPU test suite (closed forms, library reductions,
invariants and planted mistakes). One reading has nothing in the paper to pin
it to: the selection score's norm and its aggregation over layers (the paper
names the signal, KV deviation over the 2nd to 4th layers, but gives no
formula), so for ``selection_scores`` the pins check the implementation of that
reading and its parity against the paper is unpinned.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

from . import build as _build

_HERE = os.path.dirname(os.path.abspath(__file__))

_i64p = ctypes.POINTER(ctypes.c_int64)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)


def _ptr(a: np.ndarray, t):
    return a.ctypes.data_as(t)


def _rows_arg(rows, n):
    if rows is None:
        return np.arange(n, dtype=np.int64)
    return np.ascontiguousarray(np.asarray(rows, dtype=np.int64))


class Oracle:
    """Handle on one build of the oracle library.

    ``plant`` names a mistake planted in the Python composition (used only by
    the tests that show the pins have teeth): ``"no_hybrid"`` skips the
    important-row write-back, ``"no_question_kv"`` leaves the question K/V out
    of the cache, ``"fuse_shift"`` writes question outputs one row early.
    """

    def __init__(self, lib_path: str | None = None, plant: str | None = None):
        if lib_path is None:
            lib_path = _build.DEFAULT_LIB
            if not os.path.exists(lib_path):
                _build.build()
        self.lib_path = lib_path
        self.plant = plant
        lib = ctypes.CDLL(lib_path)
        lib.daf_oracle_mutant.restype = ctypes.c_int
        lib.daf_oracle_threads.restype = ctypes.c_int
        lib.daf_oracle_gather_rows.argtypes = [_u8p, ctypes.c_int64, _i64p, ctypes.c_int64, _u8p]
        lib.daf_oracle_scatter_rows.argtypes = [_u8p, ctypes.c_int64, _i64p, ctypes.c_int64, _u8p]
        lib.daf_oracle_mask_stage1.argtypes = [_i64p, ctypes.c_int64, _i64p, ctypes.c_int64, _u8p]
        lib.daf_oracle_mask_stage2.argtypes = [ctypes.c_int64, ctypes.c_int64, _i64p, ctypes.c_int64, _u8p]
        lib.daf_oracle_mask_position.argtypes = [_i64p, _i64p, ctypes.c_int64, ctypes.c_int64, _u8p]
        lib.daf_oracle_masked_attention.argtypes = [
            _f32p, _f32p, _f32p, _u8p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
            ctypes.c_int32, ctypes.c_double, _i64p, ctypes.c_int64, _f64p, _f64p, _f64p]
        lib.daf_oracle_masked_attention.restype = ctypes.c_int
        self.lib = lib
        self.mutant = lib.daf_oracle_mutant()

    @property
    def threads(self) -> int:
        """OpenMP threads the oracle's loops use."""
        return int(self.lib.daf_oracle_threads())

    # ---- byte-level row movement (Sec. 2 items 1 and 3) -------------------
    def gather_rows(self, src: np.ndarray, rows) -> np.ndarray:
        """dst[i] = src[rows[i]], byte for byte, for a 2-D (or higher) array."""
        src = np.ascontiguousarray(src)
        r = _rows_arg(rows, 0)
        row_bytes = src[0:1].nbytes if src.shape[0] else 0
        dst = np.zeros((len(r),) + src.shape[1:], dtype=src.dtype)
        if len(r):
            assert r.min() >= 0 and r.max() < src.shape[0]
            self.lib.daf_oracle_gather_rows(_ptr(src, _u8p), row_bytes, _ptr(r, _i64p), len(r),
                                            _ptr(dst, _u8p))
        return dst

    def scatter_rows(self, dst: np.ndarray, rows, src: np.ndarray) -> np.ndarray:
        """Return a copy of dst with out[rows[i]] = src[i], byte for byte."""
        out = np.array(dst, copy=True, order="C")
        src = np.ascontiguousarray(src, dtype=dst.dtype)
        r = _rows_arg(rows, 0)
        assert src.shape[0] == len(r) and src.shape[1:] == dst.shape[1:]
        if len(r):
            assert r.min() >= 0 and r.max() < dst.shape[0]
            self.lib.daf_oracle_scatter_rows(_ptr(out, _u8p), out[0:1].nbytes, _ptr(r, _i64p),
                                             len(r), _ptr(src, _u8p))
        return out

    # ---- masks ------------------------------------------------------------
    def mask_stage1(self, pos, rows=None) -> np.ndarray:
        pos = np.ascontiguousarray(np.asarray(pos, dtype=np.int64))
        n = len(pos)
        r = _rows_arg(rows, n)
        mask = np.zeros((len(r), n), dtype=np.uint8)
        if len(r) and n:
            self.lib.daf_oracle_mask_stage1(_ptr(pos, _i64p), n, _ptr(r, _i64p), len(r),
                                            _ptr(mask, _u8p))
        return mask

    def mask_stage2(self, L_d: int, L_q: int, rows=None) -> np.ndarray:
        r = _rows_arg(rows, L_q)
        mask = np.zeros((len(r), L_d + L_q), dtype=np.uint8)
        if len(r):
            self.lib.daf_oracle_mask_stage2(L_d, L_q, _ptr(r, _i64p), len(r), _ptr(mask, _u8p))
        return mask

    def mask_position(self, qpos, nk: int, rows=None) -> np.ndarray:
        qpos = np.ascontiguousarray(np.asarray(qpos, dtype=np.int64))
        r = _rows_arg(rows, len(qpos))
        mask = np.zeros((len(r), nk), dtype=np.uint8)
        if len(r) and nk:
            self.lib.daf_oracle_mask_position(_ptr(qpos, _i64p), _ptr(r, _i64p), len(r), nk,
                                              _ptr(mask, _u8p))
        return mask

    # ---- attention ----------------------------------------------------------
    def attention(self, q, k, v, mask, scale: float, rows=None, want_p: bool = False):
        """Masked scaled-dot-product attention by definition.

        q: [nq, hq, d]; k, v: [nk, hkv, d] (float32 values); mask: [nrows, nk].
        Returns o [nrows, hq, d] float64 and lse [nrows, hq] float64 (and the
        probabilities [nrows, hq, nk] if want_p).
        """
        q = np.ascontiguousarray(q, dtype=np.float32)
        k = np.ascontiguousarray(k, dtype=np.float32)
        v = np.ascontiguousarray(v, dtype=np.float32)
        mask = np.ascontiguousarray(mask, dtype=np.uint8)
        nq, hq, d = q.shape
        nk, hkv, d2 = k.shape
        assert d2 == d and v.shape == k.shape and hq % hkv == 0
        r = _rows_arg(rows, nq)
        assert mask.shape == (len(r), nk)
        o = np.zeros((len(r), hq, d), dtype=np.float64)
        lse = np.zeros((len(r), hq), dtype=np.float64)
        p = np.zeros((len(r), hq, nk), dtype=np.float64) if want_p else None
        if len(r) == 0:
            return (o, lse, p) if want_p else (o, lse)
        rc = self.lib.daf_oracle_masked_attention(
            _ptr(q, _f32p), _ptr(k, _f32p), _ptr(v, _f32p), _ptr(mask, _u8p), nk, hq, hkv, d,
            float(scale), _ptr(r, _i64p), len(r), _ptr(o, _f64p), _ptr(lse, _f64p),
            _ptr(p, _f64p) if want_p else None)
        if rc != 0:
            raise ValueError("a query row has no visible key")
        return (o, lse, p) if want_p else (o, lse)

    # ---- the three stages -------------------------------------------------
    def hybrid_kv(self, k_cache, v_cache, idx, k_imp, v_imp, k_q, v_q, L_d: int):
        """Hybrid KV cache (Sec. 2 item 2): rows idx[i] take the recomputed
        k_imp[i]/v_imp[i]; rows L_d + j take the question's k_q[j]/v_q[j].
        Caches are [L_d + L_q, hkv, d] raw arrays; returns new copies."""
        idx = np.asarray(idx, dtype=np.int64)
        L_q = k_q.shape[0]
        kh, vh = k_cache, v_cache
        if self.plant != "no_hybrid":
            kh = self.scatter_rows(kh, idx, k_imp)
            vh = self.scatter_rows(vh, idx, v_imp)
        if self.plant != "no_question_kv":
            qrows = np.arange(L_d, L_d + L_q, dtype=np.int64)
            kh = self.scatter_rows(kh, qrows, k_q)
            vh = self.scatter_rows(vh, qrows, v_q)
        return np.array(kh, copy=True), np.array(vh, copy=True)

    def stage1(self, q_imp, k_imp, v_imp, pos, scale, rows=None, want_p=False):
        """Important-token self-attention (Sec. 2 item 1): keys are the
        important tokens only, visible when not after the query in the
        original order."""
        mask = self.mask_stage1(pos, rows)
        return self.attention(q_imp, k_imp, v_imp, mask, scale, rows, want_p)

    def stage2(self, q_q, k_hyb, v_hyb, L_d, scale, rows=None, want_p=False):
        """Question-document attention (Sec. 2 item 2) over the hybrid
        [L_d + L_q] cache, question part causal."""
        L_q = q_q.shape[0]
        mask = self.mask_stage2(L_d, L_q, rows)
        return self.attention(q_q, k_hyb, v_hyb, mask, scale, rows, want_p)

    # ---- comparison patterns (Complexity Analysis) ----------------------------
    def position_attention(self, q, k, v, qpos, scale, rows=None, want_p=False):
        """Queries at original positions qpos over a key sequence, each seeing
        the keys at positions 0..qpos (causal by position)."""
        mask = self.mask_position(qpos, k.shape[0], rows)
        return self.attention(q, k, v, mask, scale, rows, want_p)

    def full_recompute(self, q, k, v, scale, rows=None):
        """Full recomputation: causal attention over every token of the
        sequence with fresh Q/K/V (the r = 1 case of the comparison)."""
        return self.position_attention(q, k, v, np.arange(q.shape[0]), scale, rows)

    def cacheblend(self, q_imp, q_q, k_hyb, v_hyb, idx, L_d: int, scale, rows=None):
        """The recomputation pattern the Complexity Analysis attributes to
        CacheBlend: the important tokens and the question tokens attend over
        the full context (the hybrid [L_d + L_q] cache), each causal by its
        original position. Rows are the important rows, then the question."""
        idx = np.asarray(idx, dtype=np.int64)
        L_q = q_q.shape[0]
        q = np.concatenate([np.asarray(q_imp, np.float32), np.asarray(q_q, np.float32)], axis=0)
        qpos = np.concatenate([idx, L_d + np.arange(L_q, dtype=np.int64)])
        return self.position_attention(q, k_hyb, v_hyb, qpos, scale, rows)

    # ---- important-token selection (Sec. 2 item 1) -----------------------------
    def selection_scores(self, k_fresh, k_cached) -> np.ndarray:
        """Per document token, the mean over the selection layers of the L2
        norm of the deviation between the freshly computed keys and the
        offline cached keys (all KV heads and features of the token).

        k_fresh, k_cached: [layers, L_d, hkv, d] float32 values. Returns
        float64 [L_d]. The paper names the signal (KV deviation, aggregated
        over several early layers, typically the 2nd to the 4th) but not the
        norm or the aggregation; this is the reading the repository takes."""
        kf = np.asarray(k_fresh, np.float64)
        kc = np.asarray(k_cached, np.float64)
        assert kf.shape == kc.shape and kf.ndim == 4
        dev = (kf - kc).reshape(kf.shape[0], kf.shape[1], -1)
        norms = np.sqrt((dev * dev).sum(axis=2))
        if self.plant == "select_one_layer":
            return norms[0]
        return norms.mean(axis=0)

    def select_important(self, scores, n: int) -> np.ndarray:
        """The n tokens with the highest scores (equal scores: lower index
        first), returned in ascending original order (the condensed sequence
        keeps the original order)."""
        scores = np.asarray(scores, np.float64)
        assert 0 <= n <= len(scores)
        ties = -np.arange(len(scores)) if self.plant == "select_tie_high" else np.arange(len(scores))
        order = np.lexsort((ties, -scores))  # score desc, then index asc
        return np.sort(order[:n]).astype(np.int64)

    def fuse_hidden(self, hidden, idx, o_imp, o_q, L_d: int):
        """State fusion (Sec. 2 item 3): hidden[idx[i]] = o_imp[i] and
        hidden[L_d + j] = o_q[j] (rows flattened to hq*d); other rows keep
        their values. All three arrays must share a dtype."""
        idx = np.asarray(idx, dtype=np.int64)
        L_q = o_q.shape[0]
        T = hidden.shape[0]
        h = hidden.reshape(T, -1)
        out = self.scatter_rows(h, idx, o_imp.reshape(len(idx), -1))
        start = L_d - 1 if self.plant == "fuse_shift" else L_d
        qrows = np.arange(start, start + L_q, dtype=np.int64)
        out = self.scatter_rows(out, qrows, o_q.reshape(L_q, -1))
        return out.reshape(hidden.shape)

    def layer(self, idx, q_imp, k_imp, v_imp, q_q, k_q, v_q, k_cache, v_cache, hidden,
              scale, L_d: int, raw_to_f32=None):
        """One DAF layer: hybrid KV, stage 1, stage 2, fusion.

        ``k_imp``... ``v_cache`` are raw arrays (moved bytewise);
        ``raw_to_f32`` widens raw arrays to float32 for the attention math
        (identity for float32 data). ``hidden`` is widened to float64 and
        the float64 stage outputs are fused into it.
        """
        w = raw_to_f32 if raw_to_f32 is not None else (lambda a: np.asarray(a, np.float32))
        k_h, v_h = self.hybrid_kv(k_cache, v_cache, idx, k_imp, v_imp, k_q, v_q, L_d)
        o_imp, lse_imp = self.stage1(w(q_imp), w(k_imp), w(v_imp), idx, scale)
        o_q, lse_q = self.stage2(w(q_q), w(k_h), w(v_h), L_d, scale)
        hid = self.fuse_hidden(np.asarray(w(hidden), np.float64), idx, o_imp, o_q, L_d)
        return dict(k_cache=k_h, v_cache=v_h, o_imp=o_imp, lse_imp=lse_imp, o_q=o_q,
                    lse_q=lse_q, hidden=hid)


def default_scale(head_dim: int) -> float:
    """Softmax scale 1/sqrt(head_dim) (standard scaled dot-product attention;
    the paper does not state one)."""
    return 1.0 / math.sqrt(head_dim)


_default = None


def get() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default
