"""GPU: every output row of both attention stages at full sizes.

With all queries zero every logit is zero, so the attention of a row is the
plain mean of the value rows it sees and its LSE is the log of their count
(a closed form, independent of the oracle's attention code). That makes every
row of a large launch checkable on the host, which the sampled-row parity
tests cannot do: a query block whose job never ran, ran twice into the wrong
rows, or ran over the wrong key range shows up here. The layouts cover the
ways the kernels deal their jobs: KV heads served by XCD pairs, by single
XCDs, or dealt round-robin over the XCDs; one request and several; the
heavy/light pairing of causal jobs on and off; head dims 128 and 64; and the
comparison patterns (queries at given positions) at the benchmark's size.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import daf_inputs as di
import oracle as orc_mod
from parity import assert_attn_close, assert_lse_close

pytestmark = pytest.mark.gpu


def _shape(name, L_d, L_q, n, hq, hkv, d=128, seed=0):
    return di.Shape(name, L_d=L_d, L_q=L_q, n=n, hq=hq, hkv=hkv, d=d, dtype=di.BF16, seed=seed)


LAYOUTS = {
    # KV head on an XCD pair, causal job pairing on (the benchmark's layer)
    "xcd_pairs_32k": [_shape("a", 32768, 128, 4915, 28, 4, seed=71)],
    # Hkv does not divide the 8 XCDs: work groups dealt round-robin, pairing on
    "round_robin": [_shape("b", 12000, 40, 11000, 12, 3, seed=72)],
    # one KV head per XCD, pairing on
    "one_head_per_xcd": [_shape("c", 9500, 50, 9000, 16, 8, seed=73)],
    # head dim 64, KV head on 4 XCDs, pairing on
    "d64": [_shape("d", 21000, 20, 20000, 8, 2, d=64, seed=74)],
    # two requests in one launch, the heavier one first
    "batch": [_shape("e", 16000, 100, 6000, 28, 4, seed=75), _shape("f", 7000, 37, 1000, 28, 4, seed=76)],
    # too few jobs for the pairing
    "unpaired": [_shape("g", 13000, 64, 2000, 28, 4, seed=77)],
}


def _running_means(v: np.ndarray, hq: int) -> np.ndarray:
    """v [rows, Hkv, D] -> [rows, Hq, D]: row i is the mean of rows 0..i, and
    query head h reads KV head h // (Hq / Hkv)."""
    c = np.cumsum(v.astype(np.float64), axis=0) / np.arange(1, v.shape[0] + 1, dtype=np.float64)[:, None, None]
    return np.repeat(c, hq // v.shape[1], axis=1)


@pytest.mark.parametrize("layout", list(LAYOUTS))
def test_zero_queries_every_row(layout):
    from paper_2607_21599_amd.tensors import LayerBuffers
    shapes = LAYOUTS[layout]
    batch = di.make_batch(shapes)
    a = batch.arrays
    a["q_imp"] = np.zeros_like(a["q_imp"])
    a["q_q"] = np.zeros_like(a["q_q"])
    s0 = shapes[0]
    buf = LayerBuffers(a, batch.cu_doc, batch.cu_q, batch.cu_imp, s0.hq, s0.hkv, s0.d)
    buf.layer()
    torch.cuda.synchronize()
    o_imp = buf["o_imp"].float().cpu().numpy()
    o_q = buf["o_q"].float().cpu().numpy()
    lse_imp = buf["lse_imp"].cpu().numpy().T
    lse_q = buf["lse_q"].cpu().numpy().T
    orc = orc_mod.get()
    for b, s in enumerate(shapes):
        r = batch.request(b)
        i0, i1 = batch.cu_imp[b], batch.cu_imp[b + 1]
        q0, q1 = batch.cu_q[b], batch.cu_q[b + 1]
        # stage 1: the important rows in original order, each over itself and the earlier ones
        exp1 = _running_means(di.raw_to_f32(r["v_imp"]), s.hq)
        assert_attn_close(o_imp[i0:i1], exp1, di.BF16, f"{layout} req {b} stage1")
        cnt1 = np.log(np.arange(1, s.n + 1, dtype=np.float64))[:, None].repeat(s.hq, axis=1)
        assert_lse_close(lse_imp[i0:i1], cnt1, di.BF16, f"{layout} req {b} stage1 lse")
        # stage 2: question row j over the hybrid cache rows 0 .. L_d + j
        _, vh = orc.hybrid_kv(r["k_cache"], r["v_cache"], r["idx"], r["k_imp"], r["v_imp"], r["k_q"], r["v_q"], s.L_d)
        exp2 = _running_means(di.raw_to_f32(vh), s.hq)[s.L_d:]
        assert_attn_close(o_q[q0:q1], exp2, di.BF16, f"{layout} req {b} stage2")
        cnt2 = np.log(s.L_d + np.arange(1, s.L_q + 1, dtype=np.float64))[:, None].repeat(s.hq, axis=1)
        assert_lse_close(lse_q[q0:q1], cnt2, di.BF16, f"{layout} req {b} stage2 lse")
        # and the fused hidden rows are the stage outputs
        hid = buf["hidden"][int(batch.cu_tok[b]):int(batch.cu_tok[b + 1])].float().cpu().numpy()
        assert np.array_equal(hid[r["idx"]].reshape(s.n, s.hq, s.d), o_imp[i0:i1]), f"{layout} req {b} hidden"
        assert np.array_equal(hid[s.L_d:].reshape(s.L_q, s.hq, s.d), o_q[q0:q1]), f"{layout} req {b} hidden q"


def test_zero_queries_every_row_patterns_32k():
    """The comparison patterns at the benchmark's size, every row: the
    CacheBlend rows (important and question tokens at their positions over the
    whole hybrid cache) and full recomputation (every token over its prefix)
    return the mean of the cache's value rows up to their position."""
    from paper_2607_21599_amd.tensors import LayerBuffers
    s = LAYOUTS["xcd_pairs_32k"][0]
    batch = di.make_batch([s])
    a = batch.arrays
    a["q_imp"] = np.zeros_like(a["q_imp"])
    a["q_q"] = np.zeros_like(a["q_q"])
    buf = LayerBuffers(a, batch.cu_doc, batch.cu_q, batch.cu_imp, s.hq, s.hkv, s.d)
    buf.fuse_kv()
    buf.prepare_patterns(np.zeros((s.T, s.hq, s.d), dtype=np.uint16))
    buf.cacheblend()
    buf.full_recompute()
    torch.cuda.synchronize()
    r = batch.request(0)
    _, vh = orc_mod.get().hybrid_kv(r["k_cache"], r["v_cache"], r["idx"], r["k_imp"], r["v_imp"], r["k_q"],
                                    r["v_q"], s.L_d)
    means = _running_means(di.raw_to_f32(vh), s.hq)
    pos = np.concatenate([r["idx"].astype(np.int64), s.L_d + np.arange(s.L_q)])
    assert_attn_close(buf["o_cb"].float().cpu().numpy(), means[pos], di.BF16, "CacheBlend pattern")
    assert_lse_close(buf["lse_cb"].cpu().numpy().T, np.log(pos + 1.0)[:, None].repeat(s.hq, axis=1), di.BF16,
                     "CacheBlend pattern lse")
    assert_attn_close(buf["o_full"].float().cpu().numpy(), means, di.BF16, "full recomputation")
    assert_lse_close(buf["lse_full"].cpu().numpy().T, np.log(np.arange(1, s.T + 1.0))[:, None].repeat(s.hq, axis=1),
                     di.BF16, "full recomputation lse")
