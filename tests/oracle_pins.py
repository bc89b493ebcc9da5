"""Pins for the CPU oracle: facts the paper and mathematics fix, checked
without re-using the oracle's own formulas.

Each pin takes an ``oracle.Oracle`` and raises AssertionError when the oracle
disagrees. The kinds of evidence:
  * reductions to a library routine: with every document token important
    (r = 1) DAF stage 1 is ordinary causal self-attention, and stage 2 is the
    last L_q rows of causal attention over the concatenated [documents;
    question] sequence (Sec. 2 items 1-2, Hardware Compatibility paragraph:
    every part is standard dense attention). torch's float64
    scaled_dot_product_attention on the CPU is the independent routine;
  * closed forms: zero queries give running means and lse = ln(count); a
    hand-worked two-token case; constant values give back the constant;
  * invariants: probability rows sum to one, exact visible-pair counts
    n(n+1)/2 and L_q*L_d + L_q(L_q+1)/2 (the exact forms behind the
    Complexity Analysis), independence from cache rows the stage must not
    read, equivariance under reordering the condensed sequence;
  * brute force over every important subset of a tiny document set.
The tests in ``test_oracle_mutants.py`` plant mistakes in the oracle and check
that at least one pin fails for each.
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import torch
import torch.nn.functional as F

TOL = 1e-10


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _randn(rng, *shape):
    return rng.standard_normal(size=shape).astype(np.float32)


def sdpa_causal(q, k, v, scale):
    """torch float64 causal SDPA, token-major [L, H, D] in and out."""
    tq = torch.from_numpy(np.asarray(q, np.float64)).permute(1, 0, 2).unsqueeze(0)
    tk = torch.from_numpy(np.asarray(k, np.float64)).permute(1, 0, 2).unsqueeze(0)
    tv = torch.from_numpy(np.asarray(v, np.float64)).permute(1, 0, 2).unsqueeze(0)
    o = F.scaled_dot_product_attention(tq, tk, tv, is_causal=True, scale=scale, enable_gqa=True)
    return o[0].permute(1, 0, 2).numpy()


def _close(a, b, tol=TOL, what=""):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    err = np.max(np.abs(a - b)) if a.size else 0.0
    assert err <= tol * max(1.0, np.max(np.abs(b)) if b.size else 1.0), f"{what}: max err {err}"


# ---------------------------------------------------------------------------
def pin_hand_two_tokens(orc):
    """Two tokens, head_dim 1, scale 1: q = (1, 1), k = (0, 1), v = (1, 3).
    Row 0 sees only key 0: o = 1, lse = 0. Row 1 sees scores (0, 1):
    o = (1 + 3e) / (1 + e), lse = ln(1 + e)."""
    q = np.array([[[1.0]], [[1.0]]], np.float32)
    k = np.array([[[0.0]], [[1.0]]], np.float32)
    v = np.array([[[1.0]], [[3.0]]], np.float32)
    o, lse = orc.stage1(q, k, v, np.array([0, 1]), 1.0)
    e = math.e
    _close(o[:, 0, 0], [1.0, (1 + 3 * e) / (1 + e)], what="hand o")
    _close(lse[:, 0], [0.0, math.log(1 + e)], what="hand lse")


def pin_stage1_full_recompute(orc):
    """r = 1: stage 1 over all document tokens is causal attention (GQA 2:1)."""
    rng = _rng(11)
    L, hq, hkv, d = 37, 4, 2, 16
    q, k, v = _randn(rng, L, hq, d), _randn(rng, L, hkv, d), _randn(rng, L, hkv, d)
    scale = 1.0 / math.sqrt(d)
    o, _ = orc.stage1(q, k, v, np.arange(L), scale)
    _close(o, sdpa_causal(q, k, v, scale), what="stage1 r=1")


def pin_stage1_condensed(orc):
    """Sparse sorted important set: stage 1 is causal attention over the
    condensed sequence (positions have gaps; only their order matters)."""
    rng = _rng(12)
    L_d, n, hq, hkv, d = 60, 17, 6, 3, 8
    pos = np.sort(rng.choice(L_d, size=n, replace=False))
    q, k, v = _randn(rng, n, hq, d), _randn(rng, n, hkv, d), _randn(rng, n, hkv, d)
    o, _ = orc.stage1(q, k, v, pos, 0.7)
    _close(o, sdpa_causal(q, k, v, 0.7), what="stage1 condensed")


def pin_stage1_position_order(orc):
    """Reordering the condensed rows (with their positions) reorders the
    outputs: visibility follows original positions, not storage order."""
    rng = _rng(13)
    n, hq, hkv, d = 19, 2, 1, 8
    pos = np.sort(rng.choice(100, size=n, replace=False))
    q, k, v = _randn(rng, n, hq, d), _randn(rng, n, hkv, d), _randn(rng, n, hkv, d)
    o, lse = orc.stage1(q, k, v, pos, 0.5)
    perm = rng.permutation(n)
    o2, lse2 = orc.stage1(q[perm], k[perm], v[perm], pos[perm], 0.5)
    _close(o2, o[perm], what="perm o")
    _close(lse2, lse[perm], what="perm lse")


def _sparse_layer_inputs(rng, L_d, L_q, n, hq, hkv, d, idx=None):
    if idx is None:
        idx = np.sort(rng.choice(L_d, size=n, replace=False))
    n = len(idx)
    T = L_d + L_q
    return dict(
        idx=np.asarray(idx, np.int64), q_imp=_randn(rng, n, hq, d), k_imp=_randn(rng, n, hkv, d),
        v_imp=_randn(rng, n, hkv, d), q_q=_randn(rng, L_q, hq, d), k_q=_randn(rng, L_q, hkv, d),
        v_q=_randn(rng, L_q, hkv, d), k_cache=_randn(rng, T, hkv, d), v_cache=_randn(rng, T, hkv, d),
        hidden=_randn(rng, T, hq * d))


def pin_hybrid_cache(orc):
    """The hybrid cache equals numpy fancy-index assignment: important rows
    take the recomputed K/V, rows L_d.. take the question K/V."""
    rng = _rng(14)
    L_d, L_q = 40, 6
    x = _sparse_layer_inputs(rng, L_d, L_q, 11, 4, 2, 8)
    kh, vh = orc.hybrid_kv(x["k_cache"], x["v_cache"], x["idx"], x["k_imp"], x["v_imp"],
                           x["k_q"], x["v_q"], L_d)
    ke, ve = x["k_cache"].copy(), x["v_cache"].copy()
    ke[x["idx"]] = x["k_imp"]
    ve[x["idx"]] = x["v_imp"]
    ke[L_d:] = x["k_q"]
    ve[L_d:] = x["v_q"]
    assert np.array_equal(kh.view(np.uint32), ke.view(np.uint32))
    assert np.array_equal(vh.view(np.uint32), ve.view(np.uint32))


def pin_stage2_concat(orc):
    """Stage 2 equals the last L_q rows of one causal attention over the
    concatenated [documents; question] sequence with the hybrid cache (the
    document rows' queries are arbitrary)."""
    rng = _rng(15)
    L_d, L_q, hq, hkv, d = 29, 7, 4, 2, 16
    x = _sparse_layer_inputs(rng, L_d, L_q, 9, hq, hkv, d)
    kh, vh = orc.hybrid_kv(x["k_cache"], x["v_cache"], x["idx"], x["k_imp"], x["v_imp"],
                           x["k_q"], x["v_q"], L_d)
    o, _ = orc.stage2(x["q_q"], kh, vh, L_d, 0.25)
    ke, ve = x["k_cache"].copy(), x["v_cache"].copy()
    ke[x["idx"]], ve[x["idx"]] = x["k_imp"], x["v_imp"]
    ke[L_d:], ve[L_d:] = x["k_q"], x["v_q"]
    q_full = np.concatenate([_randn(rng, L_d, hq, d), x["q_q"]])
    ref = sdpa_causal(q_full, ke, ve, 0.25)[L_d:]
    _close(o, ref, what="stage2 concat")


def pin_constant_values(orc):
    """Every value row equal to c: every output row is c (both stages)."""
    rng = _rng(16)
    n, L_d, L_q, hq, hkv, d = 13, 20, 5, 4, 2, 8
    c = _randn(rng, 1, hkv, d)
    q, k = _randn(rng, n, hq, d), _randn(rng, n, hkv, d)
    v = np.repeat(c, n, axis=0)
    o, _ = orc.stage1(q, k, v, np.arange(n) * 3, 0.4)
    exp = np.repeat(c, hq // hkv, axis=1)
    _close(o, np.broadcast_to(exp, o.shape), tol=1e-12, what="const v stage1")
    kc = _randn(rng, L_d + L_q, hkv, d)
    vc = np.repeat(c, L_d + L_q, axis=0)
    o2, _ = orc.stage2(_randn(rng, L_q, hq, d), kc, vc, L_d, 0.4)
    _close(o2, np.broadcast_to(exp, o2.shape), tol=1e-12, what="const v stage2")


def pin_zero_queries(orc):
    """Zero queries make every visible score 0: the output is the mean of the
    visible values and lse = ln(number of visible keys)."""
    rng = _rng(17)
    n, hq, hkv, d = 15, 2, 1, 8
    pos = np.sort(rng.choice(40, size=n, replace=False))
    q = np.zeros((n, hq, d), np.float32)
    k, v = _randn(rng, n, hkv, d), _randn(rng, n, hkv, d)
    o, lse = orc.stage1(q, k, v, pos, 0.3)
    cnt = np.arange(1, n + 1, dtype=np.float64)
    mean = np.cumsum(v.astype(np.float64), axis=0) / cnt[:, None, None]
    _close(o, np.repeat(mean, hq, axis=1), what="zero-q stage1")
    _close(lse, np.repeat(np.log(cnt)[:, None], hq, axis=1), what="zero-q lse1")
    L_d, L_q = 23, 6
    kc, vc = _randn(rng, L_d + L_q, hkv, d), _randn(rng, L_d + L_q, hkv, d)
    o2, lse2 = orc.stage2(np.zeros((L_q, hq, d), np.float32), kc, vc, L_d, 0.3)
    cnt2 = np.arange(L_d + 1, L_d + L_q + 1, dtype=np.float64)
    mean2 = np.cumsum(vc.astype(np.float64), axis=0)[L_d:] / cnt2[:, None, None]
    _close(o2, np.repeat(mean2, hq, axis=1), what="zero-q stage2")
    _close(lse2, np.repeat(np.log(cnt2)[:, None], hq, axis=1), what="zero-q lse2")


def pin_gqa_groups(orc):
    """Values constant per KV head g (= g + 1): query head h returns
    floor(h / G) + 1 with G = Hq / Hkv query heads per KV head."""
    rng = _rng(18)
    n, hq, hkv, d = 9, 6, 3, 4
    q, k = _randn(rng, n, hq, d), _randn(rng, n, hkv, d)
    v = np.zeros((n, hkv, d), np.float32)
    for g in range(hkv):
        v[:, g, :] = g + 1
    o, _ = orc.stage1(q, k, v, np.arange(n), 0.5)
    for h in range(hq):
        _close(o[:, h, :], np.full((n, d), h // (hq // hkv) + 1.0), tol=1e-12, what=f"gqa h{h}")


def pin_needle(orc):
    """A key aligned with every query and far larger than the rest takes all
    the weight from the rows that can see it (and sets their lse), and none
    from the rows before it."""
    rng = _rng(19)
    n, hq, hkv, d, j = 12, 2, 1, 8, 5
    e = np.zeros(d, np.float32)
    e[0] = 1.0
    q = np.broadcast_to(e, (n, hq, d)).copy()
    k = 0.01 * _randn(rng, n, hkv, d)
    k[j, 0] = 400.0 * e
    v = _randn(rng, n, hkv, d)
    o, lse = orc.stage1(q, k, v, np.arange(n), 1.0 / math.sqrt(d))
    for i in range(j, n):
        _close(o[i, :, :], np.broadcast_to(v[j, 0], (hq, d)), tol=1e-9, what=f"needle row {i}")
        # the needle's logit dominates the log-sum-exp: lse = 400/sqrt(d) + O(e^-100)
        _close(lse[i], np.full(hq, 400.0 / math.sqrt(d)), tol=1e-9, what=f"needle lse {i}")
    ref_before = sdpa_causal(q[:j], k[:j], v[:j], 1.0 / math.sqrt(d))
    _close(o[:j], ref_before, what="rows before needle")


def pin_probabilities(orc):
    """Probability rows sum to one, masked entries are exactly zero, and the
    visible-pair counts are n(n+1)/2 (stage 1) and L_q*L_d + L_q(L_q+1)/2
    (stage 2)."""
    rng = _rng(20)
    n, hq, hkv, d = 14, 2, 1, 8
    pos = np.sort(rng.choice(50, size=n, replace=False))
    _, _, p = orc.stage1(_randn(rng, n, hq, d), _randn(rng, n, hkv, d), _randn(rng, n, hkv, d), pos,
                         0.3, want_p=True)
    _close(p.sum(axis=2), np.ones((n, hq)), tol=1e-13, what="p1 rows")
    assert np.all(p[:, 0, :][np.triu_indices(n, 1)] == 0.0)
    assert int((p[:, 0, :] > 0).sum()) == n * (n + 1) // 2
    assert int(orc.mask_stage1(pos).sum()) == n * (n + 1) // 2
    L_d, L_q = 21, 5
    kc, vc = _randn(rng, L_d + L_q, hkv, d), _randn(rng, L_d + L_q, hkv, d)
    _, _, p2 = orc.stage2(_randn(rng, L_q, hq, d), kc, vc, L_d, 0.3, want_p=True)
    _close(p2.sum(axis=2), np.ones((L_q, hq)), tol=1e-13, what="p2 rows")
    assert int((p2[:, 0, :] > 0).sum()) == L_q * L_d + L_q * (L_q + 1) // 2
    assert int(orc.mask_stage2(L_d, L_q).sum()) == L_q * L_d + L_q * (L_q + 1) // 2
    for jq in range(L_q):
        assert np.all(p2[jq, :, L_d + jq + 1:] == 0.0)


def pin_layer_independence(orc):
    """Stage 1 reads only important tokens: changing other cache rows leaves
    o_imp unchanged. Stage 2 reads the hybrid cache: changing the offline rows
    at important positions (which the write-back replaces) leaves o_q unchanged,
    while changing any other offline row changes it."""
    rng = _rng(21)
    L_d, L_q, hq, hkv, d = 30, 4, 4, 2, 8
    x = _sparse_layer_inputs(rng, L_d, L_q, 8, hq, hkv, d)
    base = orc.layer(scale=0.35, L_d=L_d, **x)
    y = dict(x)
    y["k_cache"], y["v_cache"] = x["k_cache"].copy(), x["v_cache"].copy()
    y["k_cache"][x["idx"]] += 5.0
    y["v_cache"][x["idx"]] -= 3.0
    other = np.setdiff1d(np.arange(L_d), x["idx"])
    alt = orc.layer(scale=0.35, L_d=L_d, **y)
    _close(alt["o_imp"], base["o_imp"], tol=0.0, what="o_imp independent")
    _close(alt["o_q"], base["o_q"], tol=0.0, what="o_q reads hybrid rows")
    z = dict(x)
    z["v_cache"] = x["v_cache"].copy()
    z["v_cache"][other[0]] += 1.0
    alt2 = orc.layer(scale=0.35, L_d=L_d, **z)
    assert np.max(np.abs(alt2["o_q"] - base["o_q"])) > 1e-6, "o_q ignores an offline row"
    _close(alt2["o_imp"], base["o_imp"], tol=0.0, what="o_imp ignores offline rows")


def pin_layer_full_recompute(orc):
    """r = 1: the fused hidden state of a DAF layer equals causal attention
    over all L_d + L_q tokens (what a full recompute produces)."""
    rng = _rng(22)
    L_d, L_q, hq, hkv, d = 26, 6, 4, 2, 8
    x = _sparse_layer_inputs(rng, L_d, L_q, 0, hq, hkv, d, idx=np.arange(L_d))
    out = orc.layer(scale=0.3, L_d=L_d, **x)
    q_full = np.concatenate([x["q_imp"], x["q_q"]])
    k_full = np.concatenate([x["k_imp"], x["k_q"]])
    v_full = np.concatenate([x["v_imp"], x["v_q"]])
    ref = sdpa_causal(q_full, k_full, v_full, 0.3)
    _close(out["hidden"].reshape(L_d + L_q, hq, d), ref, what="layer r=1")


def pin_gather_scatter(orc):
    """Gather equals numpy fancy indexing; scatter equals fancy assignment and
    leaves other rows untouched; gathering scattered rows gives them back."""
    rng = _rng(23)
    src = rng.integers(0, 2**16, size=(50, 24), dtype=np.uint16)
    rows = np.sort(rng.choice(50, size=17, replace=False))
    g = orc.gather_rows(src, rows)
    assert np.array_equal(g, src[rows])
    dst = rng.integers(0, 2**16, size=(50, 24), dtype=np.uint16)
    s = orc.scatter_rows(dst, rows, g)
    ref = dst.copy()
    ref[rows] = g
    assert np.array_equal(s, ref)
    assert np.array_equal(orc.gather_rows(s, rows), g)
    keep = np.setdiff1d(np.arange(50), rows)
    assert np.array_equal(s[keep], dst[keep])


def pin_fuse_rows(orc):
    """Fusion writes o_imp[i] to hidden row idx[i], o_q[j] to row L_d + j, and
    nothing else (fancy assignment as the reference)."""
    rng = _rng(24)
    L_d, L_q, hq, d = 33, 5, 2, 4
    idx = np.sort(rng.choice(L_d, size=10, replace=False))
    hidden = _randn(rng, L_d + L_q, hq * d)
    o_imp, o_q = _randn(rng, 10, hq, d), _randn(rng, L_q, hq, d)
    out = orc.fuse_hidden(hidden, idx, o_imp, o_q, L_d)
    ref = hidden.copy()
    ref[idx] = o_imp.reshape(10, -1)
    ref[L_d:] = o_q.reshape(L_q, -1)
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))


def pin_brute_force_subsets(orc):
    """Every non-empty important subset of a 6-token document set, with a
    2-token question: stage 1 is causal attention over the chosen tokens and
    stage 2 the question rows of causal attention over [hybrid docs; question]."""
    rng = _rng(25)
    L_d, L_q, hq, hkv, d = 6, 2, 2, 1, 4
    base = _sparse_layer_inputs(rng, L_d, L_q, L_d, hq, hkv, d, idx=np.arange(L_d))
    q_doc = _randn(rng, L_d, hq, d)
    for m in range(1, L_d + 1):
        for sub in itertools.combinations(range(L_d), m):
            sub = np.array(sub)
            x = dict(base)
            x["idx"] = sub
            for key in ("q_imp", "k_imp", "v_imp"):
                x[key] = base[key][:m]
            out = orc.layer(scale=0.6, L_d=L_d, **x)
            _close(out["o_imp"], sdpa_causal(x["q_imp"], x["k_imp"], x["v_imp"], 0.6),
                   what=f"subset {sub} stage1")
            ke, ve = base["k_cache"].copy(), base["v_cache"].copy()
            ke[sub], ve[sub] = x["k_imp"], x["v_imp"]
            ke[L_d:], ve[L_d:] = base["k_q"], base["v_q"]
            ref = sdpa_causal(np.concatenate([q_doc, base["q_q"]]), ke, ve, 0.6)[L_d:]
            _close(out["o_q"], ref, what=f"subset {sub} stage2")


def _py_causal_attention(q, k, v, scale, limits, group):
    """Attention written out in plain Python floats (fp64, math module only):
    row i of query head h sees keys 0 .. limits[i] of KV head h // group.
    q: [rows][Hq][D], k, v: [keys][Hkv][D] nested lists. Returns (o, lse)."""
    d = len(q[0][0])
    out, lse = [], []
    for i, qi in enumerate(q):
        o_row, l_row = [], []
        for h, qh in enumerate(qi):
            g = h // group
            s = [scale * math.fsum(qh[t] * k[j][g][t] for t in range(d)) for j in range(limits[i] + 1)]
            m = max(s)
            e = [math.exp(x - m) for x in s]
            z = math.fsum(e)
            o_row.append([math.fsum(e[j] * v[j][g][t] for j in range(len(e))) / z for t in range(d)])
            l_row.append(m + math.log(z))
        out.append(o_row)
        lse.append(l_row)
    return out, lse


def pin_pure_python_subsets(orc):
    """Every non-empty important subset of a 7-token document set with a
    3-token question (GQA 2:1), recomputed by a second implementation in pure
    Python floats (no numpy, no torch): the hybrid cache by list assignment,
    stage 1 over the chosen tokens, stage 2 over [hybrid docs; question]. The
    C oracle must agree to 1e-12 relative, outputs and LSE."""
    rng = _rng(26)
    L_d, L_q, hq, hkv, d = 7, 3, 4, 2, 5
    base = _sparse_layer_inputs(rng, L_d, L_q, L_d, hq, hkv, d, idx=np.arange(L_d))
    scale = 0.45
    to_list = lambda a: np.asarray(a, np.float64).tolist()
    k_cache, v_cache = to_list(base["k_cache"]), to_list(base["v_cache"])
    q_q, k_q, v_q = to_list(base["q_q"]), to_list(base["k_q"]), to_list(base["v_q"])

    def rel(a, b, what):
        a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
        assert a.shape == b.shape, what
        err = float(np.max(np.abs(a - b) / np.maximum(np.abs(b), 1e-300)))
        assert err <= 1e-12, f"{what}: relative error {err:.3g}"

    for m in range(1, L_d + 1):
        for sub in itertools.combinations(range(L_d), m):
            x = dict(base)
            x["idx"] = np.array(sub)
            for key in ("q_imp", "k_imp", "v_imp"):
                x[key] = base[key][:m]
            out = orc.layer(scale=scale, L_d=L_d, **x)
            q_imp, k_imp, v_imp = to_list(x["q_imp"]), to_list(x["k_imp"]), to_list(x["v_imp"])
            o1, l1 = _py_causal_attention(q_imp, k_imp, v_imp, scale, list(range(m)), hq // hkv)
            kh = [row[:] for row in k_cache[:L_d]] + k_q
            vh = [row[:] for row in v_cache[:L_d]] + v_q
            for i, t in enumerate(sub):
                kh[t], vh[t] = k_imp[i], v_imp[i]
            o2, l2 = _py_causal_attention(q_q, kh, vh, scale, [L_d + j for j in range(L_q)], hq // hkv)
            rel(out["o_imp"], o1, f"subset {sub} stage1")
            rel(out["lse_imp"], l1, f"subset {sub} stage1 lse")
            rel(out["o_q"], o2, f"subset {sub} stage2")
            rel(out["lse_q"], l2, f"subset {sub} stage2 lse")


def pin_full_recompute_patterns(orc):
    """Comparison pattern 1 (full recomputation): causal attention over every
    token of the sequence, equal to torch's causal SDPA (GQA 7:1)."""
    rng = _rng(31)
    L, hq, hkv, d = 41, 7, 1, 16
    q, k, v = _randn(rng, L, hq, d), _randn(rng, L, hkv, d), _randn(rng, L, hkv, d)
    o, _ = orc.full_recompute(q, k, v, 0.3)
    _close(o, sdpa_causal(q, k, v, 0.3), what="full recompute")


def pin_cacheblend_rows(orc):
    """Comparison pattern 2 (the CacheBlend recomputation the Complexity
    Analysis describes): important and question tokens over the full hybrid
    context are the rows idx and L_d + j of one causal attention over the
    whole sequence whose queries at those positions are q_imp and q_q."""
    rng = _rng(32)
    L_d, L_q, hq, hkv, d = 31, 6, 4, 2, 16
    x = _sparse_layer_inputs(rng, L_d, L_q, 11, hq, hkv, d)
    kh, vh = orc.hybrid_kv(x["k_cache"], x["v_cache"], x["idx"], x["k_imp"], x["v_imp"],
                           x["k_q"], x["v_q"], L_d)
    o, _ = orc.cacheblend(x["q_imp"], x["q_q"], kh, vh, x["idx"], L_d, 0.4)
    q_full = _randn(rng, L_d + L_q, hq, d)
    q_full[x["idx"]] = x["q_imp"]
    q_full[L_d:] = x["q_q"]
    ke, ve = x["k_cache"].copy(), x["v_cache"].copy()
    ke[x["idx"]], ve[x["idx"]] = x["k_imp"], x["v_imp"]
    ke[L_d:], ve[L_d:] = x["k_q"], x["v_q"]
    ref = sdpa_causal(q_full, ke, ve, 0.4)
    rows = np.concatenate([x["idx"], L_d + np.arange(L_q)])
    _close(o, ref[rows], what="cacheblend rows")


def pin_position_zero_queries(orc):
    """Zero queries at sorted positions p: each output row is the mean of the
    value rows 0..p and lse = ln(p + 1) (closed form)."""
    rng = _rng(33)
    nk, hq, hkv, d = 23, 2, 1, 8
    v = _randn(rng, nk, hkv, d)
    k = _randn(rng, nk, hkv, d)
    qpos = np.array([0, 3, 4, 10, 22])
    q = np.zeros((len(qpos), hq, d), np.float32)
    o, lse = orc.position_attention(q, k, v, qpos, 1.0)
    for i, p in enumerate(qpos):
        for h in range(hq):
            _close(o[i, h], v[: p + 1, 0].astype(np.float64).mean(axis=0), what="position mean")
            _close(lse[i, h], math.log(p + 1), what="position lse")


def pin_selection_brute_force(orc):
    """Selection on a tiny case, against scores written out with plain loops
    and a choice by exhaustive comparison: token t is chosen iff fewer than n
    tokens beat it (higher score, or equal score and lower index)."""
    rng = _rng(51)
    layers, L, hkv, d = 3, 9, 2, 3
    kc = _randn(rng, layers, L, hkv, d)
    kf = kc + _randn(rng, layers, L, hkv, d) * rng.uniform(0.1, 2.0, size=(1, L, 1, 1)).astype(np.float32)
    sc = orc.selection_scores(kf, kc)
    for t in range(L):
        per_layer = []
        for l in range(layers):
            acc = 0.0
            for h in range(hkv):
                for j in range(d):
                    diff = float(kf[l, t, h, j]) - float(kc[l, t, h, j])
                    acc += diff * diff
            per_layer.append(math.sqrt(acc))
        _close(sc[t], sum(per_layer) / layers, what="score by loops")
    for n in range(L + 1):
        got = orc.select_important(sc, n)
        want = [t for t in range(L)
                if sum(1 for u in range(L) if sc[u] > sc[t] or (sc[u] == sc[t] and u < t)) < n]
        assert list(got) == want, f"selection n={n}: {list(got)} vs {want}"


def pin_selection_invariants(orc):
    """Scaling every deviation by a constant keeps the choice; a token whose
    keys match the cache in every layer is never chosen while tokens with a
    deviation remain; a token deviating in a single layer counts a third as
    much as the same deviation in all three (the layers are averaged); ties
    go to the lower index."""
    rng = _rng(52)
    layers, L, hkv, d = 3, 40, 2, 8
    kc = _randn(rng, layers, L, hkv, d)
    dev = _randn(rng, layers, L, hkv, d) * rng.uniform(0.1, 3.0, size=(1, L, 1, 1)).astype(np.float32)
    dev[:, 7] = 0.0
    s1 = orc.selection_scores(kc + dev, kc)
    s2 = orc.selection_scores(kc + 2 * dev, kc)
    for n in (1, 10, 39):
        assert list(orc.select_important(s1, n)) == list(orc.select_important(s2, n)), "scale"
        assert 7 not in orc.select_important(s1, n), "zero deviation chosen"
    one = np.zeros((layers, 2, 1, 4), np.float32)
    base = np.zeros_like(one)
    one[0, 0, 0, 0] = 3.0            # token 0: deviation 3 in one layer
    one[:, 1, 0, 0] = 1.0            # token 1: deviation 1 in every layer
    s = orc.selection_scores(one, base)
    _close(s, [1.0, 1.0], what="layer mean")
    assert list(orc.select_important(s, 1)) == [0], "tie to the lower index"


ALL_PINS = [
    pin_hand_two_tokens, pin_stage1_full_recompute, pin_stage1_condensed,
    pin_stage1_position_order, pin_hybrid_cache, pin_stage2_concat, pin_constant_values,
    pin_zero_queries, pin_gqa_groups, pin_needle, pin_probabilities, pin_layer_independence,
    pin_layer_full_recompute, pin_gather_scatter, pin_fuse_rows, pin_brute_force_subsets,
    pin_pure_python_subsets,
    pin_full_recompute_patterns, pin_cacheblend_rows, pin_position_zero_queries,
    pin_selection_brute_force, pin_selection_invariants,
]
