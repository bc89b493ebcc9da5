"""Shared helpers of the GPU parity tests: oracle runs on (sampled) rows and
the acceptance bar.

Acceptance (bf16 inputs, fp32 accumulation): max-abs <= 2e-2 and mean-abs
<= 2e-3 against the fp64 oracle, plus a relative Frobenius error <= 1e-2 per
head (the inputs' near-uniform softmax makes outputs small, so the absolute
bar alone would be weak). fp32 inputs: max-abs <= 1e-4, mean-abs <= 1e-5.
LSE: absolute error <= 4e-3 (bf16) / 1e-5 (fp32). The bf16 kernel rounds the
probabilities to bf16 before the P.V product (reading of the unstated
precision) and normalises by the sum of those rounded values, so the row sum it
reports differs from the exact one by at most the bf16 rounding of the terms,
a relative 2^-8 when one key dominates a row: |ln(1 + 2^-8)| = 3.9e-3.
"""
from __future__ import annotations

import numpy as np

import daf_inputs as di
import oracle as orc_mod

BF16_MAX, BF16_MEAN, BF16_REL = 2e-2, 2e-3, 1e-2
F32_MAX, F32_MEAN = 1e-4, 1e-5


def scale_of(shape) -> float:
    return orc_mod.default_scale(shape.d)


def assert_attn_close(got, ref, dtype: str, what: str):
    """got: float32 [rows, H, D] from the GPU; ref: float64 oracle output."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, f"{what}: shape {got.shape} vs {ref.shape}"
    if got.size == 0:
        return
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    err = np.abs(got - ref)
    mx, mean = float(err.max()), float(err.mean())
    if dtype == di.BF16:
        assert mx <= BF16_MAX and mean <= BF16_MEAN, f"{what}: max {mx:.3g} mean {mean:.3g}"
        num = np.sqrt(((got - ref) ** 2).sum(axis=(0, 2)))
        den = np.sqrt((ref ** 2).sum(axis=(0, 2)))
        rel = float((num / np.maximum(den, 1e-30)).max())
        assert rel <= BF16_REL, f"{what}: relative Frobenius {rel:.3g}"
    else:
        assert mx <= F32_MAX and mean <= F32_MEAN, f"{what}: max {mx:.3g} mean {mean:.3g}"


def assert_lse_close(got, ref, dtype: str, what: str):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape
    if got.size == 0:
        return
    tol = 4e-3 if dtype == di.BF16 else 1e-5
    err = float(np.abs(got - ref).max())
    assert err <= tol, f"{what}: lse max err {err:.3g}"


def sample_rows(n: int, k: int, seed: int, tile: int = 128) -> np.ndarray:
    """Up to k rows of [0, n): the ends, tile boundaries and random rows."""
    if n <= k:
        return np.arange(n)
    rng = np.random.Generator(np.random.PCG64(seed))
    must = {0, 1, n - 1, n - 2}
    for t in (tile - 1, tile, 2 * tile - 1, 2 * tile, (n // tile) * tile - 1, (n // tile) * tile):
        if 0 <= t < n:
            must.add(t)
    rest = rng.choice(n, size=max(0, k - len(must)), replace=False)
    return np.unique(np.concatenate([np.array(sorted(must)), rest]))


def oracle_request(req: dict, rows1=None, rows2=None, want=("s1", "s2")):
    """Oracle stage outputs of one request (rows1/rows2 restrict the rows)."""
    orc = orc_mod.get()
    s = req["shape"]
    sc = scale_of(s)
    w = di.raw_to_f32
    out = {}
    if "s1" in want:
        o1, l1 = orc.stage1(w(req["q_imp"]), w(req["k_imp"]), w(req["v_imp"]), req["idx"], sc, rows1)
        out["o_imp"], out["lse_imp"] = o1, l1
    if "s2" in want:
        kh, vh = orc.hybrid_kv(req["k_cache"], req["v_cache"], req["idx"], req["k_imp"], req["v_imp"],
                               req["k_q"], req["v_q"], s.L_d)
        out["k_hyb"], out["v_hyb"] = kh, vh
        o2, l2 = orc.stage2(w(req["q_q"]), w(kh), w(vh), s.L_d, sc, rows2)
        out["o_q"], out["lse_q"] = o2, l2
    return out
