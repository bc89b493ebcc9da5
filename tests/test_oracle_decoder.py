"""Pins of the decoder-layer oracle (the projections, norms, rotary embedding
and MLP around the DAF attention) against what the mathematics fixes: closed
forms, invariants and reductions, chosen so that a dropped term, a wrong sign
or a swapped index in any piece fails one of them. No formula is retyped
here."""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle as orc_mod
from oracle import decoder as dec


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


# ---- RMSNorm ---------------------------------------------------------------------
def test_rmsnorm_constant_rows_give_the_weight():
    w = _rng(1).standard_normal(16)
    for c in (3.0, -0.25):
        y = dec.rmsnorm(np.full((1, 16), c), w, 0.0)
        assert np.allclose(y[0], np.sign(c) * w, rtol=0, atol=1e-12)


def test_rmsnorm_unit_rms_scale_invariance_and_eps():
    x = _rng(2).standard_normal((5, 64))
    y = dec.rmsnorm(x, np.ones(64), 0.0)
    assert np.allclose(np.sqrt(np.mean(y * y, axis=1)), 1.0, atol=1e-12)
    assert np.allclose(dec.rmsnorm(7.5 * x, np.ones(64), 0.0), y, atol=1e-12)
    z = dec.rmsnorm(np.zeros((1, 8)), np.ones(8), 1e-6)  # a zero row stays zero, no division by zero
    assert np.all(z == 0.0)
    # eps enters under the root: a row of ones with eps = 3 scales by 1/2
    assert np.allclose(dec.rmsnorm(np.ones((1, 4)), np.ones(4), 3.0), 0.5)


# ---- linear ---------------------------------------------------------------------------
def test_linear_identity_one_hot_linearity_residual():
    rng = _rng(3)
    x = rng.standard_normal((6, 10))
    assert np.allclose(dec.linear(x, np.eye(10)), x)
    W = rng.standard_normal((7, 10))
    # a one-hot row picks the matching input column of W ([out][in] layout)
    for i in (0, 4, 9):
        e = np.zeros((1, 10))
        e[0, i] = 1.0
        assert np.allclose(dec.linear(e, W)[0], W[:, i])
    x2 = rng.standard_normal((6, 10))
    assert np.allclose(dec.linear(2.0 * x + x2, W), 2.0 * dec.linear(x, W) + dec.linear(x2, W))
    b, r = rng.standard_normal(7), rng.standard_normal((6, 7))
    assert np.allclose(dec.linear(x, W, b, r) - dec.linear(x, W), b + r)


# ---- rotary embedding --------------------------------------------------------------------
def test_rope_closed_forms():
    # D = 2: one pair at frequency theta^0 = 1, so position p rotates by p radians
    x = np.array([[[1.0, 0.0]]])
    for p in (1, 2, 5):
        y = dec.rope(x, np.array([p]), 10000.0)
        assert np.allclose(y[0, 0], [math.cos(p), math.sin(p)], atol=1e-12)
    # D = 4, theta = 100: pair 1 turns at 100^(-1/2) = 0.1 rad per position
    x = np.array([[[0.0, 1.0, 0.0, 0.0]]])  # feature 1 is the first half of pair 1
    y = dec.rope(x, np.array([10]), 100.0)
    assert np.allclose(y[0, 0], [0.0, math.cos(1.0), 0.0, math.sin(1.0)], atol=1e-12)


def test_rope_identity_norms_and_relative_positions():
    rng = _rng(4)
    q, k = rng.standard_normal((3, 2, 8)), rng.standard_normal((3, 2, 8))
    assert np.allclose(dec.rope(q, np.zeros(3), 1e4), q)
    pos = np.array([0, 7, 123])
    y = dec.rope(q, pos, 1e4)
    pairs = lambda a: a[..., :4] ** 2 + a[..., 4:] ** 2  # noqa: E731
    assert np.allclose(pairs(y), pairs(q))
    # scores depend on position differences only: shift both by 1000
    pk = np.array([3, 3, 50])
    s0 = np.sum(dec.rope(q, pos, 1e4) * dec.rope(k, pk, 1e4), axis=-1)
    s1 = np.sum(dec.rope(q, pos + 1000, 1e4) * dec.rope(k, pk + 1000, 1e4), axis=-1)
    assert np.allclose(s0, s1, atol=1e-10)


# ---- SiLU gate ------------------------------------------------------------------------------
def test_silu_mul_values_and_identity():
    assert dec.silu_mul(np.array([0.0]), np.array([5.0]))[0] == 0.0
    assert abs(dec.silu_mul(np.array([1.0]), np.array([1.0]))[0] - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15
    g = _rng(5).standard_normal(50)
    one = np.ones(50)
    assert np.allclose(dec.silu_mul(g, one) - dec.silu_mul(-g, one), g)  # silu(x) - silu(-x) = x
    assert np.allclose(dec.silu_mul(g, 3.0 * one), 3.0 * dec.silu_mul(g, one))
    assert abs(dec.silu_mul(np.array([40.0]), np.array([1.0]))[0] - 40.0) < 1e-12


# ---- the layer composition --------------------------------------------------------------
def _weights(rng, H, hq, hkv, d, inter):
    m = lambda o, i: rng.standard_normal((o, i)) / math.sqrt(i)  # noqa: E731
    return dict(w_in=1 + 0.1 * rng.standard_normal(H), wq=m(hq * d, H), bq=0.1 * rng.standard_normal(hq * d),
                wk=m(hkv * d, H), bk=0.1 * rng.standard_normal(hkv * d), wv=m(hkv * d, H),
                bv=0.1 * rng.standard_normal(hkv * d), wo=m(H, hq * d), w_post=1 + 0.1 * rng.standard_normal(H),
                wg=m(inter, H), wu=m(inter, H), wd=m(H, inter))


def test_layer_with_zero_output_projections_is_the_identity():
    rng = _rng(6)
    H, hq, hkv, d, inter, T = 32, 2, 1, 16, 48, 9
    w = _weights(rng, H, hq, hkv, d, inter)
    w["wo"][:] = 0.0
    w["wd"][:] = 0.0
    x = rng.standard_normal((T, H))
    y, _ = dec.decoder_layer(x, np.arange(T), w, dec.full_attention(orc_mod.get(), 0.25), 1e-6, 1e4, hq, hkv, d)
    assert np.array_equal(y, x)


def test_daf_layer_at_r_equal_1_is_the_full_layer():
    """With every document token important, the DAF layer (stage 1 over the
    documents, stage 2 for the question over the hybrid cache) is the full
    recomputation of the layer: same output rows, to rounding."""
    rng = _rng(7)
    H, hq, hkv, d, inter, L_d, L_q = 64, 4, 2, 16, 96, 21, 6
    T = L_d + L_q
    w = _weights(rng, H, hq, hkv, d, inter)
    x = rng.standard_normal((T, H))
    pos = np.arange(T)
    orc = orc_mod.get()
    sc = 1.0 / math.sqrt(d)
    full, _ = dec.decoder_layer(x, pos, w, dec.full_attention(orc, sc), 1e-6, 1e4, hq, hkv, d)
    # the offline cache holds arbitrary stale K/V: at r = 1 every row is replaced
    stale = rng.standard_normal((T, hkv, d))
    idx = np.arange(L_d)
    daf, _ = dec.decoder_layer(x, pos, w, dec.daf_attention(orc, idx, stale, stale, L_d, sc), 1e-6, 1e4, hq, hkv, d)
    assert np.allclose(daf, full, rtol=0, atol=1e-5)
    # and with fewer important tokens the question rows do depend on the stale cache
    idx = np.arange(0, L_d, 3)
    rows = np.concatenate([idx, np.arange(L_d, T)])
    part, _ = dec.decoder_layer(x[rows], pos[rows], w, dec.daf_attention(orc, idx, stale, stale, L_d, sc), 1e-6,
                                1e4, hq, hkv, d)
    assert not np.allclose(part[len(idx):], full[L_d:], atol=1e-3)


@pytest.mark.parametrize("plant", ["rope_sign", "rms_no_mean"])
def test_planted_mistakes_fail_the_pins(plant, monkeypatch):
    """Plant a mistake in the oracle on the CPU: a closed-form pin catches it."""
    if plant == "rope_sign":
        real = dec.rope

        def wrong(x, pos, theta):  # rotate the wrong way
            return real(x, -np.asarray(pos), theta)
        monkeypatch.setattr(dec, "rope", wrong)
        with pytest.raises(AssertionError):
            test_rope_closed_forms()
    else:
        def wrong(x, w, eps):  # sum instead of mean of squares
            x = np.asarray(x, np.float64)
            return x / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps) * w
        monkeypatch.setattr(dec, "rmsnorm", wrong)
        with pytest.raises(AssertionError):
            test_rmsnorm_unit_rms_scale_invariance_and_eps()
