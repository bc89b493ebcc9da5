"""GPU parity: every DAF entry point of libdaf.so against the CPU oracle.

Runs on an MI355X. Gather and fusion are compared bit for bit; attention
outputs and LSE against the fp64 oracle with the bar in ``parity.py``. Small
shapes are compared on every row; the 32k and batched shapes on sampled rows
(ends, 128-row tile boundaries and random rows), in the same launch
configuration the benchmark uses.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import daf_inputs as di
import oracle as orc_mod
from parity import assert_attn_close, assert_lse_close, oracle_request, sample_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2607_21599_amd as daf
    daf.lib()  # raises if libdaf.so is missing
    yield
    torch.cuda.synchronize()


def _buffers(batch: di.Batch):
    from paper_2607_21599_amd.tensors import LayerBuffers
    s = batch.shapes[0]
    return LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, s.hq, s.hkv, s.d)


def _f32(t):
    return t.detach().float().cpu().numpy()


def _raw(t):
    from paper_2607_21599_amd.tensors import to_host_raw
    return to_host_raw(t)


def _shape(name, L_d, L_q, n, hq=28, hkv=4, d=128, dtype=di.BF16, seed=0, std=0.5, sel="uniform"):
    return di.Shape(name, L_d=L_d, L_q=L_q, n=n, hq=hq, hkv=hkv, d=d, dtype=dtype, qkv_std=std,
                    cache_std=std, seed=seed, selection=sel)


SMALL = {
    "tiny_f32_1k": lambda: di.workload("tiny_f32_1k"),
    "qwen7b_6k": lambda: di.workload("qwen7b_6k"),
    "bf16_d64_gqa4": lambda: [_shape("bf16_d64", 700, 45, 230, hq=8, hkv=2, d=64, seed=31)],
    "f32_d128_gqa7": lambda: [_shape("f32_d128", 300, 17, 100, hq=14, hkv=2, d=128, dtype=di.F32,
                                     seed=32, std=1.0)],
}


# ---------------------------------------------------------------------------
# row movement: bit-exact
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", ["tiny_f32_1k", "qwen7b_6k", "qwen7b_batch8"])
def test_gather_bit_exact(name):
    import paper_2607_21599_amd as daf
    batch = di.make_batch(di.workload(name))
    buf = _buffers(batch)
    orc = orc_mod.get()
    a = batch.arrays
    # hidden rows from the full-length token layout
    dst = torch.empty((a["q_imp"].shape[0], a["hidden"].shape[1]), dtype=buf["hidden"].dtype, device="cuda")
    buf.gather_hidden(dst)
    rows_tok = np.concatenate([batch.cu_tok[b] + batch.request(b)["idx"] for b in range(len(batch.shapes))])
    exp = orc.gather_rows(a["hidden"], rows_tok)
    # K rows from a documents-only layout
    kdocs = np.concatenate([batch.request(b)["k_cache"][: batch.shapes[b].L_d] for b in range(len(batch.shapes))])
    from paper_2607_21599_amd.tensors import to_device
    kd = to_device(kdocs)
    kdst = buf.t["k_imp"].new_empty(buf.t["k_imp"].shape)
    row_bytes = kdocs[0].nbytes
    daf.daf_gather_important(buf.batch, daf.DAF_SRC_DOCS, kd, row_bytes, buf["idx"], kdst)
    rows_doc = np.concatenate([batch.cu_doc[b] + batch.request(b)["idx"] for b in range(len(batch.shapes))])
    kexp = orc.gather_rows(kdocs, rows_doc)
    torch.cuda.synchronize()
    assert np.array_equal(_raw(dst), exp)
    assert np.array_equal(_raw(kdst), kexp)


def test_gather_wide_rows():
    """Rows wider than 8 KiB (moved in column chunks) and ragged requests."""
    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import to_device
    rng = np.random.Generator(np.random.PCG64(9))
    cu_doc, cu_q, cu_imp = [0, 700, 1000, 1900], [0, 3, 3, 10], [0, 41, 41, 300]
    row_bytes = 20000
    total_tok = cu_doc[-1] + cu_q[-1]
    src = rng.integers(0, 256, size=(total_tok, row_bytes), dtype=np.uint8)
    idx = np.concatenate([np.sort(rng.choice(cu_doc[b + 1] - cu_doc[b], cu_imp[b + 1] - cu_imp[b],
                                             replace=False)) for b in range(3)]).astype(np.int32)
    b = daf.Batch(cu_doc, cu_q, cu_imp)
    s_dev = torch.from_numpy(src).cuda()
    dst = torch.zeros((cu_imp[-1], row_bytes), dtype=torch.uint8, device="cuda")
    daf.daf_gather_important(b, daf.DAF_SRC_TOKENS, s_dev, row_bytes, to_device(idx), dst)
    torch.cuda.synchronize()
    tok0 = [cu_doc[k] + cu_q[k] for k in range(3)]
    rows = np.concatenate([tok0[k] + idx[cu_imp[k]:cu_imp[k + 1]] for k in range(3)])
    assert np.array_equal(dst.cpu().numpy(), orc_mod.get().gather_rows(src, rows))


@pytest.mark.parametrize("name", ["tiny_f32_1k", "qwen7b_6k", "qwen7b_batch8"])
def test_fuse_bit_exact(name):
    """KV mode builds the hybrid cache; hidden mode scatters stage outputs
    (here: generator rows of the same shape); all other rows untouched."""
    batch = di.make_batch(di.workload(name))
    a = batch.arrays
    # use q rows as stand-in stage outputs: same shape as o_imp / o_q
    from paper_2607_21599_amd.tensors import to_device
    buf = _buffers(batch)
    buf.t["o_imp"] = to_device(a["q_imp"])
    buf.t["o_q"] = to_device(a["q_q"])
    buf.fuse_kv()
    buf.fuse_hidden()
    torch.cuda.synchronize()
    orc = orc_mod.get()
    for b in range(len(batch.shapes)):
        r = batch.request(b)
        s = batch.shapes[b]
        t0, t1 = batch.cu_tok[b], batch.cu_tok[b + 1]
        kh, vh = orc.hybrid_kv(r["k_cache"], r["v_cache"], r["idx"], r["k_imp"], r["v_imp"], r["k_q"],
                               r["v_q"], s.L_d)
        assert np.array_equal(_raw(buf["k_cache"][t0:t1]), kh), f"k_cache request {b}"
        assert np.array_equal(_raw(buf["v_cache"][t0:t1]), vh), f"v_cache request {b}"
        hexp = orc.fuse_hidden(r["hidden"], r["idx"], r["q_imp"], r["q_q"], s.L_d)
        assert np.array_equal(_raw(buf["hidden"][t0:t1]), hexp), f"hidden request {b}"


def test_check_indices():
    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import to_device
    batch = di.make_batch(di.workload("qwen7b_batch8"))
    b = daf.Batch(batch.cu_doc, batch.cu_q, batch.cu_imp)
    bad = torch.full((1,), -7, dtype=torch.int32, device="cuda")
    idx = batch.arrays["idx"].copy()
    daf.daf_check_indices(b, to_device(idx), bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == 0
    i0 = batch.cu_imp[3]
    idx[i0 + 5] = idx[i0 + 4]          # duplicate
    idx[batch.cu_imp[5]] = -1          # out of range
    idx[batch.cu_imp[8] - 1] = batch.shapes[7].L_d  # past the end
    daf.daf_check_indices(b, to_device(idx), bad)
    torch.cuda.synchronize()
    assert int(bad.item()) == 3


# ---------------------------------------------------------------------------
# attention stages
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("name", list(SMALL))
def test_stages_small_all_rows(name):
    batch = di.make_batch(SMALL[name]())
    buf = _buffers(batch)
    buf.fuse_kv()
    buf.stage1()
    buf.stage2()
    torch.cuda.synchronize()
    r = batch.request(0)
    ref = oracle_request(r)
    dt = batch.dtype
    assert_attn_close(_f32(buf["o_imp"]), ref["o_imp"], dt, "stage1")
    assert_lse_close(_f32(buf["lse_imp"]).T, ref["lse_imp"], dt, "stage1 lse")
    assert_attn_close(_f32(buf["o_q"]), ref["o_q"], dt, "stage2")
    assert_lse_close(_f32(buf["lse_q"]).T, ref["lse_q"], dt, "stage2 lse")


@pytest.mark.parametrize("n", [1, 2, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 257, 400])
def test_stage1_edge_sizes(n):
    s = _shape(f"edge_n{n}", L_d=2 * n + 3, L_q=1, n=n, hq=7, hkv=1, seed=100 + n)
    batch = di.make_batch(s)
    buf = _buffers(batch)
    buf.stage1()
    torch.cuda.synchronize()
    ref = oracle_request(batch.request(0), want=("s1",))
    assert_attn_close(_f32(buf["o_imp"]), ref["o_imp"], di.BF16, f"stage1 n={n}")
    assert_lse_close(_f32(buf["lse_imp"]).T, ref["lse_imp"], di.BF16, f"stage1 lse n={n}")


@pytest.mark.parametrize("L_d,L_q", [(0, 5), (1, 1), (100, 1), (63, 64), (500, 129), (4096, 200),
                                     (3000, 256), (20000, 7)])
def test_stage2_edge_sizes(L_d, L_q):
    n = min(L_d, 17)
    s = _shape(f"edge_{L_d}_{L_q}", L_d=L_d, L_q=L_q, n=n, hq=14, hkv=2, seed=200 + L_q)
    batch = di.make_batch(s)
    buf = _buffers(batch)
    buf.fuse_kv()
    buf.stage2()
    torch.cuda.synchronize()
    ref = oracle_request(batch.request(0), want=("s2",))
    assert_attn_close(_f32(buf["o_q"]), ref["o_q"], di.BF16, f"stage2 {L_d}/{L_q}")
    assert_lse_close(_f32(buf["lse_q"]).T, ref["lse_q"], di.BF16, f"stage2 lse {L_d}/{L_q}")


@pytest.mark.parametrize("name", ["qwen7b_16k_r05", "qwen7b_16k_r15", "qwen7b_16k_r30", "qwen7b_32k",
                                  "qwen7b_32k_lq32", "qwen7b_128k_r30"])
def test_layer_large_sampled(name):
    """Full-size layer through daf_layer_attn, oracle on sampled rows."""
    batch = di.make_batch(di.workload(name))
    buf = _buffers(batch)
    buf.layer()
    torch.cuda.synchronize()
    r = batch.request(0)
    s = batch.shapes[0]
    rows1 = sample_rows(s.n, 40, seed=1)
    rows2 = sample_rows(s.L_q, 16, seed=2)
    ref = oracle_request(r, rows1, rows2)
    assert_attn_close(_f32(buf["o_imp"])[rows1], ref["o_imp"], di.BF16, f"{name} stage1")
    assert_lse_close(_f32(buf["lse_imp"]).T[rows1], ref["lse_imp"], di.BF16, f"{name} lse1")
    assert_attn_close(_f32(buf["o_q"])[rows2], ref["o_q"], di.BF16, f"{name} stage2")
    assert_lse_close(_f32(buf["lse_q"]).T[rows2], ref["lse_q"], di.BF16, f"{name} lse2")
    # hybrid cache bit-exact, fused hidden rows equal the stage outputs bit for bit
    assert np.array_equal(_raw(buf["k_cache"]), ref["k_hyb"])
    assert np.array_equal(_raw(buf["v_cache"]), ref["v_hyb"])
    hid = buf["hidden"]
    idx_t = torch.from_numpy(r["idx"].astype(np.int64)).cuda()
    assert torch.equal(hid[idx_t].view(-1), buf["o_imp"].reshape(-1))
    assert torch.equal(hid[s.L_d:].reshape(-1), buf["o_q"].reshape(-1))
    keep = np.setdiff1d(np.arange(s.L_d), r["idx"])
    sel = np.sort(np.random.Generator(np.random.PCG64(3)).choice(keep, 256, replace=False))
    assert np.array_equal(_raw(hid[torch.from_numpy(sel).cuda()]), r["hidden"][sel])


def test_layer_small_full_oracle():
    """daf_layer_attn on the 6k layer: hidden equals the oracle's fused state
    (fused rows within tolerance, all other rows unchanged)."""
    batch = di.make_batch(di.workload("qwen7b_6k"))
    buf = _buffers(batch)
    buf.layer()
    torch.cuda.synchronize()
    r = batch.request(0)
    s = batch.shapes[0]
    ref = orc_mod.get().layer(r["idx"], r["q_imp"], r["k_imp"], r["v_imp"], r["q_q"], r["k_q"], r["v_q"],
                              r["k_cache"], r["v_cache"], r["hidden"], scale=orc_mod.default_scale(s.d),
                              L_d=s.L_d, raw_to_f32=di.raw_to_f32)
    hid = _f32(buf["hidden"])
    fused = np.concatenate([r["idx"], np.arange(s.L_d, s.T)])
    assert_attn_close(hid[fused].reshape(-1, s.hq, s.d), ref["hidden"][fused].reshape(-1, s.hq, s.d),
                      di.BF16, "fused rows")
    keep = np.setdiff1d(np.arange(s.T), fused)
    assert np.array_equal(_raw(buf["hidden"])[keep], r["hidden"][keep])


def test_layer_equals_stage_calls():
    """The one-layer driver (both stages in one grid) gives the same bits as
    the stage-by-stage calls."""
    batch = di.make_batch(di.workload("qwen7b_6k"))
    a, b = _buffers(batch), _buffers(batch)
    a.layer()
    b.fuse_kv()
    b.stage1()
    b.stage2()
    b.fuse_hidden()
    torch.cuda.synchronize()
    for k in ("o_imp", "o_q", "lse_imp", "lse_q", "hidden", "k_cache", "v_cache"):
        assert torch.equal(a[k], b[k]), k


def test_batched_ragged():
    """Eight ragged requests in one call: every request against the oracle on
    sampled rows."""
    batch = di.make_batch(di.workload("qwen7b_batch8"))
    buf = _buffers(batch)
    buf.layer()
    torch.cuda.synchronize()
    o_imp, o_q = _f32(buf["o_imp"]), _f32(buf["o_q"])
    lse_imp, lse_q = _f32(buf["lse_imp"]).T, _f32(buf["lse_q"]).T
    for b in range(len(batch.shapes)):
        r = batch.request(b)
        s = batch.shapes[b]
        rows1 = sample_rows(s.n, 12, seed=10 + b)
        rows2 = sample_rows(s.L_q, 6, seed=20 + b)
        ref = oracle_request(r, rows1, rows2)
        i0, q0 = batch.cu_imp[b], batch.cu_q[b]
        assert_attn_close(o_imp[i0 + rows1], ref["o_imp"], di.BF16, f"req {b} stage1")
        assert_lse_close(lse_imp[i0 + rows1], ref["lse_imp"], di.BF16, f"req {b} lse1")
        assert_attn_close(o_q[q0 + rows2], ref["o_q"], di.BF16, f"req {b} stage2")
        assert_lse_close(lse_q[q0 + rows2], ref["lse_q"], di.BF16, f"req {b} lse2")


def test_batch_with_empty_requests():
    shapes = [_shape("e0", 300, 20, 0, hq=7, hkv=1, seed=41), _shape("e1", 0, 9, 0, hq=7, hkv=1, seed=42),
              _shape("e2", 500, 0, 77, hq=7, hkv=1, seed=43), _shape("e3", 260, 33, 130, hq=7, hkv=1, seed=44)]
    batch = di.make_batch(shapes)
    buf = _buffers(batch)
    buf.layer()
    torch.cuda.synchronize()
    o_imp, o_q = _f32(buf["o_imp"]), _f32(buf["o_q"])
    for b, s in enumerate(shapes):
        ref = oracle_request(batch.request(b))
        i0, i1, q0, q1 = batch.cu_imp[b], batch.cu_imp[b + 1], batch.cu_q[b], batch.cu_q[b + 1]
        assert_attn_close(o_imp[i0:i1], ref["o_imp"], di.BF16, f"req {b} stage1")
        assert_attn_close(o_q[q0:q1], ref["o_q"], di.BF16, f"req {b} stage2")


def test_peaked_softmax():
    """Queries scaled by 8 (exact in bf16): logits with std ~2, a peaked
    softmax where absolute errors are not vacuous."""
    batch = di.make_batch(di.workload("qwen7b_6k"))
    for k in ("q_imp", "q_q"):
        batch.arrays[k] = di.f32_to_bf16_bits(di.raw_to_f32(batch.arrays[k]) * np.float32(8.0))
    buf = _buffers(batch)
    buf.layer()
    torch.cuda.synchronize()
    s = batch.shapes[0]
    rows1 = sample_rows(s.n, 200, seed=5)
    ref = oracle_request(batch.request(0), rows1)
    assert_attn_close(_f32(buf["o_imp"])[rows1], ref["o_imp"], di.BF16, "peaked stage1")
    assert_attn_close(_f32(buf["o_q"]), ref["o_q"], di.BF16, "peaked stage2")


def test_running_max_raised_late():
    """Keys whose logits jump far above every earlier one (by ~40 in log2
    units per step), placed well below the diagonal: the kernel forms a full
    tile's probabilities against the running max as it stands and must catch
    the overflow, raise the max, rescale and form the tile again, in stage 1
    and in stage 2 (where the loud keys reach the hybrid cache through the
    important rows, plus one offline cache row). A last key ~10 units above
    the max is formed against the old max (probability ~2^10, bf16-rounded),
    which the LSE bar covers."""
    shape = _shape("loud_keys", 3000, 40, 900, hq=8, hkv=2, d=128, seed=41)
    batch = di.make_batch([shape])
    a = batch.arrays
    d, hkv = shape.d, shape.hkv
    u = np.full(d, 1.0 / np.sqrt(d), np.float32)
    for k in ("q_imp", "q_q"):
        q = di.raw_to_f32(a[k]) + np.float32(8.0) * u
        a[k] = di.f32_to_bf16_bits(q)
    k_imp, v_imp = di.raw_to_f32(a["k_imp"]), di.raw_to_f32(a["v_imp"])
    # three keys each ~40 log2 units above the last (the max is raised), then
    # one ~10 units above (formed against the old max: its probability ~2^10)
    for j, (pos, beta) in enumerate(((100, 40.0), (300, 80.0), (500, 120.0), (700, 130.0))):
        k_imp[pos] = np.float32(beta) * u
        v_imp[pos] = np.float32(j + 1)
    a["k_imp"], a["v_imp"] = di.f32_to_bf16_bits(k_imp), di.f32_to_bf16_bits(v_imp)
    idx = a["idx"][: shape.n]
    free = np.setdiff1d(np.arange(shape.L_d - 200), idx)
    k_cache, v_cache = di.raw_to_f32(a["k_cache"]), di.raw_to_f32(a["v_cache"])
    k_cache[free[-1]] = np.float32(160.0) * u
    v_cache[free[-1]] = np.float32(4.0)
    a["k_cache"], a["v_cache"] = di.f32_to_bf16_bits(k_cache), di.f32_to_bf16_bits(v_cache)
    assert k_imp.shape[1:] == (hkv, d)
    buf = _buffers(batch)
    buf.layer()
    torch.cuda.synchronize()
    ref = oracle_request(batch.request(0))
    assert_attn_close(_f32(buf["o_imp"]), ref["o_imp"], di.BF16, "loud keys stage1")
    assert_attn_close(_f32(buf["o_q"]), ref["o_q"], di.BF16, "loud keys stage2")
    assert_lse_close(_f32(buf["lse_imp"]).T, ref["lse_imp"], di.BF16, "loud keys stage1 lse")
    assert_lse_close(_f32(buf["lse_q"]).T, ref["lse_q"], di.BF16, "loud keys stage2 lse")
    # the loud keys dominate: each row returns the value of the loudest key it sees
    o1 = _f32(buf["o_imp"])
    assert np.allclose(o1[600:700], 3.0, atol=2e-2)
    assert np.allclose(o1[704:], 4.0, atol=2e-2)


def test_repeat_runs_bit_identical():
    batch = di.make_batch(di.workload("qwen7b_16k_r15"))
    buf = _buffers(batch)
    buf.fuse_kv()
    buf.stage1()
    buf.stage2()
    first = {k: buf[k].clone() for k in ("o_imp", "o_q", "lse_imp", "lse_q")}
    for _ in range(2):
        buf.stage1()
        buf.stage2()
    torch.cuda.synchronize()
    for k, v in first.items():
        assert torch.equal(buf[k], v), k


def test_invalid_arguments_enqueue_nothing():
    import paper_2607_21599_amd as daf
    batch = di.make_batch(di.workload("tiny_f32_1k"))
    buf = _buffers(batch)
    before = buf["o_imp"].clone()
    bad = daf.AttnCfg(4, 3, 64, daf.DAF_F32)
    with pytest.raises(daf.DafError) as e:
        daf.daf_imp_self_attn(bad, buf.batch, buf["q_imp"], buf["k_imp"], buf["v_imp"], buf["o_imp"])
    assert e.value.status == 1
    with pytest.raises(daf.DafError) as e:
        daf.daf_qdoc_attn(buf.cfg, buf.batch, buf["q_q"], buf["k_cache"], buf["v_cache"], buf["o_q"], None,
                          buf["ws"], 16)
    assert e.value.status == 4
    torch.cuda.synchronize()
    assert torch.equal(before, buf["o_imp"])
