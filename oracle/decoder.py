"""Oracle for the rest of the DAF layer: the projections, norms and MLP that
surround the attention in a decoder layer.

TEST INFRASTRUCTURE ONLY, like the rest of this package: only the test suite,
the smoke check and the benchmark's CPU-baseline leg may use it.

The paper runs DAF on Qwen2.5-7B (Sec. 3) and says which rows each layer
recomputes: the QKV computation phase covers the important and question tokens
only (Sec. 2 item 2), and the fused compact state of those rows is what the
next layer's QKV computation consumes (Sec. 2 item 3). It does not restate the
model's layer; the reading taken here is the Qwen2 pre-norm decoder layer:

    h  = RMSNorm(x) * w_in
    q, k, v = h Wq^T + bq, h Wk^T + bk, h Wv^T + bv
    q, k   = RoPE(q, pos), RoPE(k, pos)          (rotate-half pairs, base theta)
    o  = attention(q, k, v)                        (DAF stages, or full causal)
    x1 = x + o Wo^T
    h2 = RMSNorm(x1) * w_post
    x2 = x1 + (SiLU(h2 Wg^T) * (h2 Wu^T)) Wd^T

Everything is plain numpy in float64; inputs are float arrays (bf16 values
widened by the caller). The attention step is passed in, so the same
composition serves the DAF layer (active rows only) and full recomputation
(every row).
"""
from __future__ import annotations

import numpy as np


def rmsnorm(x, w, eps: float):
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    x = np.asarray(x, np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * np.asarray(w, np.float64)


def linear(x, W, b=None, residual=None):
    """x W^T (+ b) (+ residual); W is [out][in]."""
    y = np.asarray(x, np.float64) @ np.asarray(W, np.float64).T
    if b is not None:
        y = y + np.asarray(b, np.float64)
    if residual is not None:
        y = y + np.asarray(residual, np.float64)
    return y


def rope(x, pos, theta: float):
    """Rotary position embedding of x [rows][heads][D] at positions pos[rows]:
    feature pairs (i, i + D/2) rotate by pos * theta^(-2i/D)."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    half = d // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / d)
    ang = np.asarray(pos, np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu_mul(g, u):
    """SiLU(g) * u, SiLU(g) = g / (1 + exp(-g))."""
    g = np.asarray(g, np.float64)
    return g / (1.0 + np.exp(-g)) * np.asarray(u, np.float64)


def decoder_layer(x, pos, wts: dict, attention, eps: float, theta: float, hq: int, hkv: int, d: int):
    """The layer above on the rows of x [rows][H] at positions pos[rows].

    ``wts``: w_in, wq, bq, wk, bk, wv, bv, wo, w_post, wg, wu, wd (float
    arrays, [out][in] for the projections). ``attention(q, k, v)`` takes the
    roped q [rows][hq][d], k and v [rows][hkv][d] and returns o [rows][hq][d]
    (the caller decides which keys each row sees). Returns (x2, parts) with
    the intermediate tensors in ``parts``."""
    rows = x.shape[0]
    h = rmsnorm(x, wts["w_in"], eps)
    q = linear(h, wts["wq"], wts["bq"]).reshape(rows, hq, d)
    k = linear(h, wts["wk"], wts["bk"]).reshape(rows, hkv, d)
    v = linear(h, wts["wv"], wts["bv"]).reshape(rows, hkv, d)
    q, k = rope(q, pos, theta), rope(k, pos, theta)
    o = attention(q, k, v).reshape(rows, hq * d)
    x1 = linear(o, wts["wo"], residual=x)
    h2 = rmsnorm(x1, wts["w_post"], eps)
    m = silu_mul(linear(h2, wts["wg"]), linear(h2, wts["wu"]))
    x2 = linear(m, wts["wd"], residual=x1)
    return x2, dict(h=h, q=q, k=k, v=v, o=o, x1=x1, h2=h2, m=m)


def daf_attention(orc, idx, k_cache, v_cache, L_d: int, scale: float):
    """attention(q, k, v) for the DAF layer of one request, rows being the n
    important rows (in idx order) then the L_q question rows: the hybrid cache
    takes the fresh K/V of the important rows at their positions and the
    question's after the documents (Sec. 2 item 2), then stage 1 and stage 2
    (Sec. 2 items 1 and 2). ``orc`` is an Oracle; k_cache / v_cache are the
    request's [L_d + L_q][hkv][d] float arrays (offline document rows)."""
    idx = np.asarray(idx, np.int64)

    def attn(q, k, v):
        n = len(idx)
        kh = np.array(k_cache, np.float64, copy=True)
        vh = np.array(v_cache, np.float64, copy=True)
        kh[idx], vh[idx] = k[:n], v[:n]
        kh[L_d:], vh[L_d:] = k[n:], v[n:]
        f = np.float32
        o1 = orc.stage1(q[:n].astype(f), k[:n].astype(f), v[:n].astype(f), idx, scale)[0]
        o2 = orc.stage2(q[n:].astype(f), kh.astype(f), vh.astype(f), L_d, scale)[0]
        return np.concatenate([o1, o2])
    return attn


def full_attention(orc, scale: float):
    """attention(q, k, v) of full recomputation: causal over every row."""
    def attn(q, k, v):
        f = np.float32
        return orc.full_recompute(q.astype(f), k.astype(f), v.astype(f), scale)[0]
    return attn
