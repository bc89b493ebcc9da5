"""GPU parity of important-token selection (daf_select_important) against the
CPU oracle. Scores are compared within the fp32 accumulation error; the chosen
indices bit for bit wherever the oracle's n-th and (n+1)-th scores are apart
by more than that error, and otherwise checked for validity (count, order,
range, nothing chosen clearly below anything left out)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import daf_inputs as di
import oracle as orc_mod

pytestmark = pytest.mark.gpu
SCORE_REL = 2e-5


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2607_21599_amd as daf
    daf.lib()
    yield
    torch.cuda.synchronize()


def _run(batch, fresh_reqs, cached_reqs, n_layers):
    """fresh_reqs / cached_reqs: per request [layers, L_d, hkv, d] raw arrays."""
    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import to_device
    s = batch.shapes[0]
    fresh = [to_device(np.ascontiguousarray(np.concatenate([f[l] for f in fresh_reqs]))) for l in range(n_layers)]
    cached = [to_device(np.ascontiguousarray(np.concatenate([c[l] for c in cached_reqs]))) for l in range(n_layers)]
    rows = int(batch.cu_doc[-1])
    scores = torch.full((max(rows, 1),), -1.0, dtype=torch.float32, device="cuda")
    idx = torch.full((max(int(batch.cu_imp[-1]), 1),), -7, dtype=torch.int32, device="cuda")
    cfg = daf.AttnCfg(s.hq, s.hkv, s.d, daf.DAF_BF16 if s.dtype == di.BF16 else daf.DAF_F32)
    daf.daf_select_important(cfg, daf.Batch(batch.cu_doc, batch.cu_q, batch.cu_imp), fresh, cached, scores, idx)
    torch.cuda.synchronize()
    return scores.cpu().numpy()[:rows], idx.cpu().numpy()


def _check(batch, fresh_reqs, cached_reqs, scores, idx):
    orc = orc_mod.get()
    w = di.raw_to_f32
    for b in range(len(batch.shapes)):
        d0, d1 = int(batch.cu_doc[b]), int(batch.cu_doc[b + 1])
        i0, i1 = int(batch.cu_imp[b]), int(batch.cu_imp[b + 1])
        n = i1 - i0
        ref = orc.selection_scores(w(fresh_reqs[b]), w(cached_reqs[b]))
        got = scores[d0:d1].astype(np.float64)
        err = np.abs(got - ref) / np.maximum(ref.max(), 1e-30)
        assert err.max() <= SCORE_REL, f"request {b}: score rel err {err.max():.3g}"
        sel = idx[i0:i1].astype(np.int64)
        want = orc.select_important(ref, n)
        assert len(sel) == n
        if n == 0:
            continue
        assert np.all(np.diff(sel) > 0) and sel[0] >= 0 and sel[-1] < d1 - d0, f"request {b}: bad order/range"
        srt = np.sort(ref)[::-1]
        gap = srt[n - 1] - (srt[n] if n < len(srt) else -np.inf)
        tol = 4 * SCORE_REL * max(ref.max(), 1e-30)
        if gap > tol:
            assert np.array_equal(sel, want), f"request {b}: selection differs from the oracle"
        else:  # near-tie at the boundary: the choice must be valid
            out = np.setdiff1d(np.arange(d1 - d0), sel)
            assert ref[sel].min() >= ref[out].max() - tol, f"request {b}: invalid near-tie choice"


@pytest.mark.parametrize("name", ["tiny_f32_1k", "qwen7b_6k", "qwen7b_32k", "qwen7b_batch8"])
def test_select_parity(name):
    shapes = di.workload(name)
    batch = di.make_batch(shapes)
    pairs = [di.make_selection_inputs(s, 3) for s in shapes]
    fresh, cached = [p[0] for p in pairs], [p[1] for p in pairs]
    scores, idx = _run(batch, fresh, cached, 3)
    _check(batch, fresh, cached, scores, idx)


@pytest.mark.parametrize("n_layers", [1, 4])
def test_select_all_and_ties(n_layers):
    """n = L_d keeps everything; exact ties (zero deviation) go to the lowest
    indices."""
    s = di.Shape("sel_ties", L_d=3000, L_q=5, n=700, hq=8, hkv=2, d=64, seed=77)
    fresh, cached = di.make_selection_inputs(s, n_layers)
    rng = np.random.Generator(np.random.PCG64(5))
    dev_rows = np.sort(rng.choice(s.L_d, size=400, replace=False))
    keep = np.zeros(s.L_d, bool)
    keep[dev_rows] = True
    fresh = np.where(keep[None, :, None, None], fresh, cached)  # only 400 tokens deviate
    for n in (700, s.L_d, 400, 1):
        sh = di.Shape("sel_ties", L_d=s.L_d, L_q=5, n=n, hq=8, hkv=2, d=64, seed=77)
        batch = di.Batch([sh], {}, np.array([0, sh.L_d]), np.array([0, 5]), np.array([0, n]))
        scores, idx = _run(batch, [fresh], [cached], n_layers)
        _check(batch, [fresh], [cached], scores, idx)
        got = idx[:n]
        if n >= 400:
            zeros = np.setdiff1d(np.arange(sh.L_d), dev_rows)[: n - 400]
            assert np.array_equal(got, np.union1d(dev_rows, zeros)), f"n={n}: ties not to the lowest indices"


def test_select_long_request_ties_across_slabs():
    """A request longer than the keys one workgroup holds in registers (a
    40000-token document beside a 5000-token one): only 300 tokens deviate,
    so the kept zero-score ties run across slab boundaries in index order."""
    rng = np.random.Generator(np.random.PCG64(11))
    shs, fresh_l, cached_l = [], [], []
    for L, n in ((40000, 20000), (5000, 900)):
        s = di.Shape("sel_long", L_d=L, L_q=3, n=n, hq=2, hkv=1, d=64, seed=91 + L)
        f, c = di.make_selection_inputs(s, 1)
        dev = np.sort(rng.choice(L, size=300, replace=False))
        keep = np.zeros(L, bool)
        keep[dev] = True
        fresh_l.append(np.where(keep[None, :, None, None], f, c))
        cached_l.append(c)
        shs.append((s, dev))
    for n0 in (20000, 39000, 300, 1):
        sh = [di.Shape("sel_long", L_d=40000, L_q=3, n=n0, hq=2, hkv=1, d=64, seed=1), shs[1][0]]
        cu_imp = np.array([0, n0, n0 + sh[1].n])
        batch = di.Batch(sh, {}, np.array([0, 40000, 45000]), np.array([0, 3, 6]), cu_imp)
        scores, idx = _run(batch, fresh_l, cached_l, 1)
        _check(batch, fresh_l, cached_l, scores, idx)
        got = idx[:n0]
        dev = shs[0][1]
        want = np.union1d(dev, np.setdiff1d(np.arange(40000), dev)[: n0 - 300]) if n0 >= 300 else None
        if want is not None:
            assert np.array_equal(got, want), f"n={n0}: ties across slabs not to the lowest indices"


def test_select_all_scores_equal():
    """No token deviates: every score is 0 and the first n tokens are kept."""
    s = di.Shape("sel_flat", L_d=2500, L_q=2, n=123, hq=2, hkv=1, d=64, seed=5)
    _, c = di.make_selection_inputs(s, 2)
    batch = di.Batch([s], {}, np.array([0, s.L_d]), np.array([0, 2]), np.array([0, s.n]))
    scores, idx = _run(batch, [c.copy()], [c], 2)
    assert np.all(scores == 0.0)
    assert np.array_equal(idx[: s.n], np.arange(s.n))
