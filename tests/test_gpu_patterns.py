"""GPU parity of the comparison patterns (daf_position_attn) against the CPU
oracle: queries at given positions of a key sequence, the CacheBlend pattern
(important and question rows over the whole hybrid cache) and full
recomputation (every token over its prefix)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import daf_inputs as di
import oracle as orc_mod
from parity import assert_attn_close, assert_lse_close, sample_rows, scale_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2607_21599_amd as daf
    daf.lib()
    yield
    torch.cuda.synchronize()


def _f32(t):
    return t.detach().float().cpu().numpy()


@pytest.mark.parametrize("n_rows,n_keys,hq,hkv,d,dtype", [
    (1, 1, 7, 1, 128, di.BF16), (5, 300, 7, 1, 128, di.BF16), (200, 1000, 28, 4, 128, di.BF16),
    (129, 129, 8, 2, 64, di.BF16), (333, 2049, 8, 2, 64, di.BF16), (97, 640, 4, 1, 64, di.F32),
    (150, 150, 14, 2, 128, di.F32)])
def test_position_attn_all_rows(n_rows, n_keys, hq, hkv, d, dtype):
    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import to_device
    rng = np.random.Generator(np.random.PCG64(n_rows * 7 + n_keys))
    pos = np.sort(rng.choice(n_keys, size=n_rows, replace=False)).astype(np.int32)
    pos[-1] = n_keys - 1 if n_rows == n_keys else pos[-1]
    q = di._normal(rng, (n_rows, hq, d), 0.5, dtype)
    k = di._normal(rng, (n_keys, hkv, d), 0.5, dtype)
    v = di._normal(rng, (n_keys, hkv, d), 0.5, dtype)
    tq, tk, tv, tp = to_device(q), to_device(k), to_device(v), to_device(pos)
    o = torch.zeros_like(tq)
    lse = torch.zeros((hq, n_rows), dtype=torch.float32, device="cuda")
    cfg = daf.AttnCfg(hq, hkv, d, daf.DAF_BF16 if dtype == di.BF16 else daf.DAF_F32)
    daf.daf_position_attn(cfg, n_rows, n_keys, tq, tp, tk, tv, o, lse)
    torch.cuda.synchronize()
    orc = orc_mod.get()
    w = di.raw_to_f32
    ro, rl = orc.position_attention(w(q), w(k), w(v), pos, orc_mod.default_scale(d))
    assert_attn_close(_f32(o), ro, dtype, "position")
    assert_lse_close(lse.cpu().numpy().T, rl, dtype, "position")


@pytest.mark.parametrize("n_rows,n_keys", [(64, 64), (300, 300), (100, 700)])
def test_position_attn_null_is_bottom_right_causal(n_rows, n_keys):
    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import to_device
    hq, hkv, d = 7, 1, 128
    rng = np.random.Generator(np.random.PCG64(n_rows + 5 * n_keys))
    q = di._normal(rng, (n_rows, hq, d), 0.5, di.BF16)
    k = di._normal(rng, (n_keys, hkv, d), 0.5, di.BF16)
    v = di._normal(rng, (n_keys, hkv, d), 0.5, di.BF16)
    tq, tk, tv = to_device(q), to_device(k), to_device(v)
    o = torch.zeros_like(tq)
    daf.daf_position_attn(daf.AttnCfg(hq, hkv, d, daf.DAF_BF16), n_rows, n_keys, tq, None, tk, tv, o)
    torch.cuda.synchronize()
    pos = np.arange(n_rows) + (n_keys - n_rows)
    w = di.raw_to_f32
    ro, _ = orc_mod.get().position_attention(w(q), w(k), w(v), pos, orc_mod.default_scale(d))
    assert_attn_close(_f32(o), ro, di.BF16, "bottom-right causal")


def _pattern_buffers(name):
    from paper_2607_21599_amd.tensors import LayerBuffers
    batch = di.make_batch(di.workload(name))
    s = batch.shapes[0]
    buf = LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, s.hq, s.hkv, s.d)
    buf.fuse_kv()
    return batch, s, buf


def test_cacheblend_6k_all_rows():
    batch, s, buf = _pattern_buffers("qwen7b_6k")
    buf.prepare_patterns()
    buf.cacheblend()
    torch.cuda.synchronize()
    req = batch.request(0)
    orc = orc_mod.get()
    w = di.raw_to_f32
    kh, vh = orc.hybrid_kv(req["k_cache"], req["v_cache"], req["idx"], req["k_imp"], req["v_imp"],
                           req["k_q"], req["v_q"], s.L_d)
    ro, rl = orc.cacheblend(w(req["q_imp"]), w(req["q_q"]), w(kh), w(vh), req["idx"], s.L_d, scale_of(s))
    assert_attn_close(_f32(buf["o_cb"]), ro, di.BF16, "cacheblend 6k")
    assert_lse_close(buf["lse_cb"].cpu().numpy().T, rl, di.BF16, "cacheblend 6k")


def test_patterns_32k_sampled():
    batch, s, buf = _pattern_buffers("qwen7b_32k")
    q_full = di.make_full_queries(s)
    buf.prepare_patterns(q_full)
    buf.cacheblend()
    buf.full_recompute()
    torch.cuda.synchronize()
    req = batch.request(0)
    orc = orc_mod.get()
    w = di.raw_to_f32
    kh, vh = orc.hybrid_kv(req["k_cache"], req["v_cache"], req["idx"], req["k_imp"], req["v_imp"],
                           req["k_q"], req["v_q"], s.L_d)
    kh, vh = w(kh), w(vh)
    rows = sample_rows(s.n + s.L_q, 48, seed=41)
    ro, _ = orc.cacheblend(w(req["q_imp"]), w(req["q_q"]), kh, vh, req["idx"], s.L_d, scale_of(s), rows)
    assert_attn_close(_f32(buf["o_cb"])[rows], ro, di.BF16, "cacheblend 32k")
    rows = sample_rows(s.T, 40, seed=42)
    ro, _ = orc.full_recompute(w(q_full), kh, vh, scale_of(s), rows)
    assert_attn_close(_f32(buf["o_full"])[rows], ro, di.BF16, "full recompute 32k")
