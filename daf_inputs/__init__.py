"""Seeded synthetic inputs for one DAF attention layer (or a ragged batch).

This module holds no attention arithmetic. It draws the tensors a DAF layer
receives (important-token indices, fresh Q/K/V of the important and question
tokens, the offline document KV cache, and a hidden-state buffer) and hands the
same values to the CPU oracle and to the HIP library.

Shapes follow Qwen2.5-7B (28 query heads, 4 KV heads, head_dim 128), the model
the paper evaluates on; a tiny fp32 shape serves correctness tests. Values are
N(0, 1) * std in float32, rounded to bfloat16 (round to nearest even) for
bfloat16 workloads; the oracle receives those exact bfloat16 values widened to
float32. Document boundaries are metadata only: the important tokens are drawn
from all documents together.

Draw order per request: important set, q_imp, k_imp, v_imp, q_q, k_q, v_q,
k_cache[:L_d], v_cache[:L_d], then fills for the cache's question rows and for
the hidden buffer (random finite bit patterns; the fusion overwrites the rows
it owns and must leave the rest untouched).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

BF16 = "bf16"
F32 = "f32"


# ---------------------------------------------------------------------------
# bfloat16 bit conversion (input preparation only)
# ---------------------------------------------------------------------------
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16, nearest-even; returns uint16 bit patterns.
    Inputs are finite (normal draws), so no NaN handling is needed."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to the float32 values they encode."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def raw_to_f32(raw: np.ndarray) -> np.ndarray:
    """float32 view of a raw buffer: bf16 bits (uint16) are widened, float32 passes."""
    if raw.dtype == np.uint16:
        return bf16_bits_to_f32(raw)
    return np.asarray(raw, dtype=np.float32)


def n_important(r: float, L_d: int) -> int:
    """Number of important tokens for fraction r: r*L_d rounded to nearest,
    halves away from zero (0.15*1024 -> 154, 0.15*32768 -> 4915)."""
    return int(math.floor(r * L_d + 0.5))


# ---------------------------------------------------------------------------
# shapes
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class Shape:
    name: str
    L_d: int
    L_q: int
    n: int
    hq: int = 28
    hkv: int = 4
    d: int = 128
    dtype: str = BF16
    qkv_std: float = 0.5
    cache_std: float = 0.5
    selection: str = "uniform"  # "uniform" without replacement, or "topk" of N(0,1) scores
    seed: int = 0
    doc_lens: tuple = field(default=())

    @property
    def T(self) -> int:
        return self.L_d + self.L_q


def _docs(L_d: int, doc: int) -> tuple:
    return tuple([doc] * (L_d // doc) + ([L_d % doc] if L_d % doc else []))


def tiny_f32() -> Shape:
    """4 documents x 256 tokens, 32 question tokens, r = 0.15, 4 query heads /
    1 KV head, head_dim 64, float32, N(0,1) values."""
    return Shape("tiny_f32_1k", L_d=1024, L_q=32, n=n_important(0.15, 1024), hq=4, hkv=1, d=64,
                 dtype=F32, qkv_std=1.0, cache_std=1.0, seed=1000, doc_lens=_docs(1024, 256))


def qwen_6k() -> Shape:
    """Qwen2.5-7B-shaped layer: 6 documents x 1024 tokens, 64 question tokens, r = 0.15."""
    return Shape("qwen7b_6k", L_d=6144, L_q=64, n=n_important(0.15, 6144), seed=2000,
                 doc_lens=_docs(6144, 1024))


def qwen_16k(r: float) -> Shape:
    """16 documents x 1024 tokens, 128 question tokens; the important set is the
    top r*L_d tokens of a seeded N(0,1) per-token score."""
    ri = {0.05: 0, 0.15: 1, 0.30: 2}[r]
    return Shape(f"qwen7b_16k_r{int(round(r * 100)):02d}", L_d=16384, L_q=128,
                 n=n_important(r, 16384), selection="topk", seed=3000 + 10 * ri,
                 doc_lens=_docs(16384, 1024))


def qwen_32k(L_q: int = 128) -> Shape:
    """Long-context layer: 32 documents x 1024 tokens, r = 0.15 (4915 important
    tokens), 128 question tokens. L_q = 32 gives the bandwidth-bound variant."""
    name = "qwen7b_32k" if L_q == 128 else f"qwen7b_32k_lq{L_q}"
    return Shape(name, L_d=32768, L_q=L_q, n=n_important(0.15, 32768), seed=4000 + (L_q != 128),
                 doc_lens=_docs(32768, 1024))


def qwen_128k() -> Shape:
    """LongBench-scale layer: L_d = 131072, r = 0.30, 128 question tokens."""
    return Shape("qwen7b_128k_r30", L_d=131072, L_q=128, n=n_important(0.30, 131072), seed=6000,
                 doc_lens=_docs(131072, 1024))


def qwen_batch8() -> list:
    """Eight independent requests: L_d = 4096*(b+1), documents of 512..2048
    tokens, L_q uniform in [32, 256], r = 0.15."""
    rng = np.random.Generator(np.random.PCG64(5000))
    lq = rng.integers(32, 257, size=8)
    shapes = []
    for b in range(8):
        L_d = 4096 * (b + 1)
        docs, left = [], L_d
        while left > 0:
            x = int(rng.integers(512, 2049))
            if left - x < 512:
                x = left
            docs.append(x)
            left -= x
        shapes.append(Shape(f"qwen7b_batch8_req{b}", L_d=L_d, L_q=int(lq[b]),
                            n=n_important(0.15, L_d), seed=5000 + b, doc_lens=tuple(docs)))
    return shapes


def workload(name: str) -> list:
    """Named workloads as lists of request shapes (a batch of one for single layers)."""
    table = {
        "tiny_f32_1k": lambda: [tiny_f32()],
        "qwen7b_6k": lambda: [qwen_6k()],
        "qwen7b_16k_r05": lambda: [qwen_16k(0.05)],
        "qwen7b_16k_r15": lambda: [qwen_16k(0.15)],
        "qwen7b_16k_r30": lambda: [qwen_16k(0.30)],
        "qwen7b_32k": lambda: [qwen_32k()],
        "qwen7b_32k_lq32": lambda: [qwen_32k(32)],
        "qwen7b_128k_r30": lambda: [qwen_128k()],
        "qwen7b_batch8": qwen_batch8,
    }
    return table[name]()


# ---------------------------------------------------------------------------
# generation
# ---------------------------------------------------------------------------
def _normal(rng, shape, std, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x) if dtype == BF16 else x


def _fill(rng, shape, dtype):
    if dtype == BF16:
        return rng.integers(0, 0x7F00, size=shape, dtype=np.uint16)
    return rng.integers(0, 0x7F000000, size=shape, dtype=np.uint32).view(np.float32)


def important_set(rng, s: Shape) -> np.ndarray:
    if s.selection == "topk":
        score = rng.standard_normal(size=s.L_d, dtype=np.float32)
        # higher score first, lower index on ties, then ascending order
        order = np.lexsort((np.arange(s.L_d), -score))
        idx = np.sort(order[: s.n])
    else:
        idx = np.sort(rng.choice(s.L_d, size=s.n, replace=False))
    return idx.astype(np.int32)


def make_request(s: Shape) -> dict:
    """All inputs of one request, raw (uint16 bf16 bits or float32)."""
    rng = np.random.Generator(np.random.PCG64(s.seed))
    r = {"shape": s}
    r["idx"] = important_set(rng, s)
    r["q_imp"] = _normal(rng, (s.n, s.hq, s.d), s.qkv_std, s.dtype)
    r["k_imp"] = _normal(rng, (s.n, s.hkv, s.d), s.qkv_std, s.dtype)
    r["v_imp"] = _normal(rng, (s.n, s.hkv, s.d), s.qkv_std, s.dtype)
    r["q_q"] = _normal(rng, (s.L_q, s.hq, s.d), s.qkv_std, s.dtype)
    r["k_q"] = _normal(rng, (s.L_q, s.hkv, s.d), s.qkv_std, s.dtype)
    r["v_q"] = _normal(rng, (s.L_q, s.hkv, s.d), s.qkv_std, s.dtype)
    kc = np.empty((s.T, s.hkv, s.d), dtype=np.uint16 if s.dtype == BF16 else np.float32)
    vc = np.empty_like(kc)
    kc[: s.L_d] = _normal(rng, (s.L_d, s.hkv, s.d), s.cache_std, s.dtype)
    vc[: s.L_d] = _normal(rng, (s.L_d, s.hkv, s.d), s.cache_std, s.dtype)
    kc[s.L_d:] = _fill(rng, (s.L_q, s.hkv, s.d), s.dtype)
    vc[s.L_d:] = _fill(rng, (s.L_q, s.hkv, s.d), s.dtype)
    r["k_cache"], r["v_cache"] = kc, vc
    r["hidden"] = _fill(rng, (s.T, s.hq * s.d), s.dtype)
    return r


def make_full_queries(s: Shape) -> np.ndarray:
    """Queries for every token of a request ([T, hq, d], raw), for the
    full-recomputation comparison pattern: drawn from their own stream
    (seed + 7919) with the request's query distribution."""
    rng = np.random.Generator(np.random.PCG64(s.seed + 7919))
    return _normal(rng, (s.T, s.hq, s.d), s.qkv_std, s.dtype)


def make_selection_inputs(s: Shape, n_layers: int = 3):
    """Keys of the selection layers for every document token: the offline
    cached keys and the freshly computed ones, [n_layers, L_d, hkv, d] raw
    each. The fresh keys deviate from the cached ones by N(0,1) noise scaled
    per token by a log-normal factor (exp(N(0, 0.5)) * 0.1), so that some
    tokens deviate much more than others. Drawn from their own stream (seed +
    104729)."""
    rng = np.random.Generator(np.random.PCG64(s.seed + 104729))
    shape = (n_layers, s.L_d, s.hkv, s.d)
    cached = rng.standard_normal(size=shape, dtype=np.float32) * np.float32(s.cache_std)
    scale = (np.exp(rng.standard_normal(size=(1, s.L_d, 1, 1)) * 0.5) * 0.1).astype(np.float32)
    fresh = cached + rng.standard_normal(size=shape, dtype=np.float32) * scale
    if s.dtype == BF16:
        return f32_to_bf16_bits(fresh), f32_to_bf16_bits(cached)
    return fresh, cached


@dataclass
class Batch:
    """Requests concatenated along the token axis, with prefix offsets.

    Row blocks: important rows by cu_imp, question rows by cu_q, cache and
    hidden rows by cu_tok (= cu_doc + cu_q, request b owns T_b rows, its
    documents first and its question last)."""
    shapes: list
    arrays: dict
    cu_doc: np.ndarray
    cu_q: np.ndarray
    cu_imp: np.ndarray

    @property
    def cu_tok(self) -> np.ndarray:
        return self.cu_doc + self.cu_q

    @property
    def dtype(self) -> str:
        return self.shapes[0].dtype

    def request(self, b: int) -> dict:
        """Views of request b's slices (idx stays request-local)."""
        a = self.arrays
        i0, i1 = self.cu_imp[b], self.cu_imp[b + 1]
        q0, q1 = self.cu_q[b], self.cu_q[b + 1]
        t0, t1 = self.cu_tok[b], self.cu_tok[b + 1]
        return dict(shape=self.shapes[b], idx=a["idx"][i0:i1], q_imp=a["q_imp"][i0:i1],
                    k_imp=a["k_imp"][i0:i1], v_imp=a["v_imp"][i0:i1], q_q=a["q_q"][q0:q1],
                    k_q=a["k_q"][q0:q1], v_q=a["v_q"][q0:q1], k_cache=a["k_cache"][t0:t1],
                    v_cache=a["v_cache"][t0:t1], hidden=a["hidden"][t0:t1])


def make_batch(shapes) -> Batch:
    if isinstance(shapes, Shape):
        shapes = [shapes]
    shapes = list(shapes)
    assert len({(s.hq, s.hkv, s.d, s.dtype) for s in shapes}) == 1
    reqs = [make_request(s) for s in shapes]
    keys = ["idx", "q_imp", "k_imp", "v_imp", "q_q", "k_q", "v_q", "k_cache", "v_cache", "hidden"]
    if len(reqs) == 1:
        arrays = {k: reqs[0][k] for k in keys}
    else:
        arrays = {k: np.concatenate([r[k] for r in reqs], axis=0) for k in keys}
    z = np.zeros(1, dtype=np.int64)
    cu_doc = np.concatenate([z, np.cumsum([s.L_d for s in shapes])]).astype(np.int32)
    cu_q = np.concatenate([z, np.cumsum([s.L_q for s in shapes])]).astype(np.int32)
    cu_imp = np.concatenate([z, np.cumsum([s.n for s in shapes])]).astype(np.int32)
    return Batch(shapes, arrays, cu_doc, cu_q, cu_imp)


def with_seed(s: Shape, seed: int, **kw) -> Shape:
    return replace(s, seed=seed, **kw)


# ---- decoder-layer inputs (projections, norms, MLP around the attention) -------

@dataclass
class ModelShape:
    """A decoder layer's widths (Qwen2.5-7B: hidden 3584, 28/4 heads of 128,
    MLP 18944, RMSNorm eps 1e-6, RoPE base 1e6)."""
    hidden: int = 3584
    hq: int = 28
    hkv: int = 4
    d: int = 128
    inter: int = 18944
    eps: float = 1e-6
    theta: float = 1e6


QWEN7B = ModelShape()
TINY_MODEL = ModelShape(hidden=256, hq=4, hkv=2, d=64, inter=512)


def make_linear_case(M: int, N: int, K: int, seed: int, bias: bool = True, residual: bool = True):
    """A [M][K] ~ N(0,1), W [N][K] ~ N(0, 1/K) (outputs of order 1), bias ~
    N(0, 0.1^2), residual ~ N(0,1); all bf16 bit patterns."""
    rng = np.random.Generator(np.random.PCG64(seed))
    A = f32_to_bf16_bits(rng.standard_normal((M, K), dtype=np.float32))
    W = f32_to_bf16_bits(rng.standard_normal((N, K), dtype=np.float32) * np.float32(1.0 / np.sqrt(K)))
    b = f32_to_bf16_bits(rng.standard_normal(N, dtype=np.float32) * np.float32(0.1)) if bias else None
    R = f32_to_bf16_bits(rng.standard_normal((M, N), dtype=np.float32)) if residual else None
    return A, W, b, R


def make_layer_weights(m: ModelShape, seed: int) -> dict:
    """Random weights of one decoder layer (bf16 bit patterns): projections
    ~ N(0, 1/fan_in) so activations stay of order 1, biases ~ N(0, 0.1^2),
    norm weights ~ 1 + N(0, 0.1^2). Projections are [out][in]."""
    rng = np.random.Generator(np.random.PCG64(seed))

    def mat(o, i):
        return f32_to_bf16_bits(rng.standard_normal((o, i), dtype=np.float32) * np.float32(1.0 / np.sqrt(i)))

    def vec(n, mean, std):
        return f32_to_bf16_bits(np.float32(mean) + rng.standard_normal(n, dtype=np.float32) * np.float32(std))

    H, q, kv = m.hidden, m.hq * m.d, m.hkv * m.d
    return dict(w_in=vec(H, 1.0, 0.1), wq=mat(q, H), bq=vec(q, 0.0, 0.1), wk=mat(kv, H), bk=vec(kv, 0.0, 0.1),
                wv=mat(kv, H), bv=vec(kv, 0.0, 0.1), wo=mat(H, q), w_post=vec(H, 1.0, 0.1),
                wg=mat(m.inter, H), wu=mat(m.inter, H), wd=mat(H, m.inter))
