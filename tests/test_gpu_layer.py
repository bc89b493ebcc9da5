"""GPU parity of the decoder-layer pieces around the attention (projections,
norms, rotary embedding, MLP gate) against the CPU oracle.

Outputs are bf16 of order-1 values: the bar is the output rounding, half a
bf16 ulp (2^-9 relative) plus fp32 accumulation error, checked as
|gpu - oracle| <= 2^-8 |oracle| + 2e-3."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import daf_inputs as di
from oracle import decoder as dec

pytestmark = pytest.mark.gpu
REL, ABS = 2.0 ** -8, 2e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2607_21599_amd as daf
    daf.lib()
    yield
    torch.cuda.synchronize()


def _dev(raw):
    from paper_2607_21599_amd.tensors import to_device
    return to_device(raw)


def _f(t):
    return t.float().cpu().numpy().astype(np.float64)


def _close(got, ref, what):
    got, ref = np.asarray(got, np.float64), np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    bound = REL * np.abs(ref) + ABS
    bad = err > bound
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} beyond the bf16 bar, worst {err.max():.3g}"


@pytest.mark.parametrize("M,N,K,bias,res", [(300, 256, 192, True, True), (77, 128, 64, False, False),
                                           (1, 384, 128, True, False), (513, 128, 640, False, True)])
def test_linear(M, N, K, bias, res):
    import paper_2607_21599_amd as daf
    A, W, b, R = di.make_linear_case(M, N, K, seed=M + N + K, bias=bias, residual=res)
    w = di.raw_to_f32
    ref = dec.linear(w(A), w(W), None if b is None else w(b), None if R is None else w(R))
    # C has 5 extra sentinel rows that must stay untouched; the residual is C itself
    C = torch.full((M + 5, N), 7.0, dtype=torch.bfloat16, device="cuda")
    if res:
        C[:M] = _dev(R)
    daf.daf_linear(M, N, K, _dev(A), _dev(W), None if b is None else _dev(b), C if res else None, C)
    torch.cuda.synchronize()
    _close(_f(C[:M]), ref, f"linear {M}x{N}x{K}")
    assert torch.all(C[M:] == 7.0), "rows past M were written"


@pytest.mark.parametrize("M,N,K,res", [(5043, 4608, 3584, False), (5043, 3584, 18944, False),
                                       (5043, 37888, 3584, False), (2100, 14848, 512, True)])
def test_linear_full_size_sampled(M, N, K, res):
    """The layer's QKV, down and gate+up projections at the 32k shape
    (n + L_q = 5043 rows; gate+up and the last case take the 256 x 256 tile,
    the last one with a ragged M and an in-place residual), oracle on sampled
    rows."""
    import paper_2607_21599_amd as daf
    A, W, b, R = di.make_linear_case(M, N, K, seed=N + K, bias=True, residual=res)
    C = _dev(R) if res else torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    daf.daf_linear(M, N, K, _dev(A), _dev(W), _dev(b), C if res else None, C)
    torch.cuda.synchronize()
    rows = np.sort(np.random.Generator(np.random.PCG64(1)).choice(M, 24, replace=False))
    rows = np.union1d(rows, [0, 255, 256, M - 1])
    w = di.raw_to_f32
    ref = dec.linear(w(A[rows]), w(W), w(b), w(R[rows]) if res else None)
    _close(_f(C[torch.from_numpy(rows).cuda()]), ref, f"linear {M}x{N}x{K}")


def test_rmsnorm_rope_silu():
    import paper_2607_21599_amd as daf
    rng = np.random.Generator(np.random.PCG64(11))
    bits = di.f32_to_bf16_bits
    w = di.raw_to_f32
    # RMSNorm over 3584-wide rows (a ragged 4-row workgroup tail)
    x = bits(rng.standard_normal((301, 3584), dtype=np.float32) * np.float32(2.0))
    g = bits(np.float32(1.0) + rng.standard_normal(3584, dtype=np.float32) * np.float32(0.1))
    y = torch.empty((301, 3584), dtype=torch.bfloat16, device="cuda")
    daf.daf_rmsnorm(301, 3584, _dev(x), _dev(g), 1e-6, y)
    # RoPE in place on the q part of q|k|v rows, positions up to 131071
    rows, hq, d = 257, 28, 128
    qkv = bits(rng.standard_normal((rows, 4608), dtype=np.float32))
    pos = np.sort(rng.choice(131072, rows, replace=False)).astype(np.int32)
    t = _dev(qkv)
    daf.daf_rope(rows, hq, d, 4608, t, _dev(pos), 1e6)
    # SiLU gate over gate|up rows
    gu = bits(rng.standard_normal((70, 2 * 512), dtype=np.float32) * np.float32(3.0))
    m = torch.empty((70, 512), dtype=torch.bfloat16, device="cuda")
    daf.daf_silu_mul(70, 512, _dev(gu), m)
    torch.cuda.synchronize()
    _close(_f(y), dec.rmsnorm(w(x), w(g), 1e-6), "rmsnorm")
    ref = dec.rope(w(qkv)[:, :hq * d].reshape(rows, hq, d), pos, 1e6).reshape(rows, hq * d)
    got = _f(t)
    _close(got[:, :hq * d], ref, "rope")
    assert np.array_equal(di.f32_to_bf16_bits(got[:, hq * d:].astype(np.float32)), qkv[:, hq * d:]), \
        "rope touched the k|v part"
    _close(_f(m), dec.silu_mul(w(gu)[:, :512], w(gu)[:, 512:]), "silu_mul")


def _layer_setup(model, L_d, L_q, n, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    bits = di.f32_to_bf16_bits
    T = L_d + L_q
    x = bits(rng.standard_normal((T, model.hidden), dtype=np.float32))
    kc = bits(rng.standard_normal((T, model.hkv, model.d), dtype=np.float32) * np.float32(0.5))
    vc = bits(rng.standard_normal((T, model.hkv, model.d), dtype=np.float32) * np.float32(0.5))
    idx = np.sort(rng.choice(L_d, n, replace=False)).astype(np.int32)
    wts = di.make_layer_weights(model, seed + 1)
    return x, kc, vc, idx, wts


def _weights_on_gpu(model, wts):
    import paper_2607_21599_amd as daf
    t = {k: _dev(v) for k, v in wts.items() if k not in ("wg", "wu")}
    t["wgu"] = _dev(np.concatenate([wts["wg"], wts["wu"]]))
    return daf.LayerWeights.from_tensors(t, model.hidden, model.inter, model.eps, model.theta)


def _oracle_weights(wts):
    return {k: di.raw_to_f32(v) for k, v in wts.items()}


def _layer_close(got, ref, what):
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    assert rel <= 1e-2 and err.max() <= 5e-2, f"{what}: rel Frobenius {rel:.3g}, max abs {err.max():.3g}"


@pytest.mark.parametrize("model,L_d,L_q,n", [(di.TINY_MODEL, 600, 32, 90), (di.TINY_MODEL, 333, 7, 333),
                                             (di.QWEN7B, 6144, 64, 922), (di.QWEN7B, 16384, 128, 2458)])
def test_decoder_layer_daf(model, L_d, L_q, n):
    """One DAF layer: only the important and question rows are recomputed;
    the hybrid cache receives their roped K/V; the output is the compact
    state (x of those rows after the layer). At the Qwen2.5-7B widths the
    projections cut their tail tiles along k (986 rows: every tile, in pieces;
    2586 rows: 512 whole tiles, then 76 in 6 pieces each, then the sum)."""
    import paper_2607_21599_amd as daf
    from oracle import get as oracle_get
    x, kc, vc, idx, wts = _layer_setup(model, L_d, L_q, n, seed=L_d + n)
    rows = np.concatenate([idx, np.arange(L_d, L_d + L_q)]).astype(np.int32)
    cfg = daf.AttnCfg(model.hq, model.hkv, model.d, daf.DAF_BF16)
    batch = daf.Batch.single(L_d, L_q, n)
    w = _weights_on_gpu(model, wts)
    xa, kd, vd, pos = _dev(x[rows]), _dev(kc), _dev(vc), _dev(rows)
    ws_bytes = daf.daf_decoder_layer_workspace_size(cfg, w, batch, daf.DAF_LAYER_DAF)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    daf.daf_decoder_layer(cfg, w, batch, daf.DAF_LAYER_DAF, _dev(idx), pos, xa, kd, vd, ws, ws_bytes)
    torch.cuda.synchronize()
    f = di.raw_to_f32
    orc = oracle_get()
    ref, parts = dec.decoder_layer(f(x[rows]), rows, _oracle_weights(wts),
                                   dec.daf_attention(orc, idx, f(kc), f(vc), L_d, 1.0 / np.sqrt(model.d)),
                                   model.eps, model.theta, model.hq, model.hkv, model.d)
    _layer_close(_f(xa), ref, f"DAF layer {L_d}/{L_q}/{n}")
    # hybrid cache: fresh roped K/V at the recomputed rows, every other row untouched
    kg = _f(kd)
    _layer_close(kg[rows], parts["k"], "hybrid K rows")
    keep = np.setdiff1d(np.arange(L_d), idx)
    assert np.array_equal(di.f32_to_bf16_bits(kg[keep].astype(np.float32)), kc[keep])


def test_decoder_layer_full():
    """Full recomputation of the layer: every row, causal over the request."""
    import paper_2607_21599_amd as daf
    from oracle import get as oracle_get
    model, L_d, L_q = di.TINY_MODEL, 500, 20
    x, _, _, _, wts = _layer_setup(model, L_d, L_q, 1, seed=5)
    T = L_d + L_q
    cfg = daf.AttnCfg(model.hq, model.hkv, model.d, daf.DAF_BF16)
    batch = daf.Batch.single(L_d, L_q, 0)
    w = _weights_on_gpu(model, wts)
    xa, pos = _dev(x), _dev(np.arange(T, dtype=np.int32))
    ws_bytes = daf.daf_decoder_layer_workspace_size(cfg, w, batch, daf.DAF_LAYER_FULL)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    daf.daf_decoder_layer(cfg, w, batch, daf.DAF_LAYER_FULL, None, pos, xa, None, None, ws, ws_bytes)
    torch.cuda.synchronize()
    ref, _ = dec.decoder_layer(di.raw_to_f32(x), np.arange(T), _oracle_weights(wts),
                               dec.full_attention(oracle_get(), 1.0 / np.sqrt(model.d)),
                               model.eps, model.theta, model.hq, model.hkv, model.d)
    _layer_close(_f(xa), ref, "full layer")


def test_decoder_layer_full_large_tiles_sampled():
    """Full recomputation at the Qwen2.5-7B widths with 9300 rows: q_proj,
    o_proj and the down projection take the 256 x 256 tile (518 tiles: two
    whole rounds of 256, then 6 tail tiles cut along k, then the sum). The
    oracle computes K/V for every row and the rest of the layer on sampled
    rows, including rows of the tail tiles (M-tiles 32-36)."""
    import paper_2607_21599_amd as daf
    from oracle import get as oracle_get
    model, L_d, L_q = di.QWEN7B, 9236, 64
    x, _, _, _, wts = _layer_setup(model, L_d, L_q, 1, seed=9)
    T = L_d + L_q
    cfg = daf.AttnCfg(model.hq, model.hkv, model.d, daf.DAF_BF16)
    batch = daf.Batch.single(L_d, L_q, 0)
    w = _weights_on_gpu(model, wts)
    xa, pos = _dev(x), _dev(np.arange(T, dtype=np.int32))
    ws_bytes = daf.daf_decoder_layer_workspace_size(cfg, w, batch, daf.DAF_LAYER_FULL)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    daf.daf_decoder_layer(cfg, w, batch, daf.DAF_LAYER_FULL, None, pos, xa, None, None, ws, ws_bytes)
    torch.cuda.synchronize()
    rng = np.random.Generator(np.random.PCG64(11))
    rows = np.union1d(rng.choice(T, 24, replace=False), rng.choice(np.arange(8192, T), 12, replace=False))
    rows = np.union1d(rows, [0, 255, 256, 8191, 8192, T - 1])
    f, ow = di.raw_to_f32, _oracle_weights(wts)
    xf = f(x)
    h = dec.rmsnorm(xf, ow["w_in"], model.eps)
    k = dec.rope(dec.linear(h, ow["wk"], ow["bk"]).reshape(T, model.hkv, model.d), np.arange(T), model.theta)
    v = dec.linear(h, ow["wv"], ow["bv"]).reshape(T, model.hkv, model.d)
    q = dec.rope(dec.linear(h[rows], ow["wq"], ow["bq"]).reshape(len(rows), model.hq, model.d), rows, model.theta)
    o = oracle_get().position_attention(q.astype(np.float32), k.astype(np.float32), v.astype(np.float32), rows,
                                        1.0 / np.sqrt(model.d))[0].reshape(len(rows), -1)
    x1 = dec.linear(o, ow["wo"], residual=xf[rows])
    h2 = dec.rmsnorm(x1, ow["w_post"], model.eps)
    ref = dec.linear(dec.silu_mul(dec.linear(h2, ow["wg"]), dec.linear(h2, ow["wu"])), ow["wd"], residual=x1)
    _layer_close(_f(xa[torch.from_numpy(rows).cuda()]), ref, "full layer, 256 x 256 tiles, sampled rows")


@pytest.mark.parametrize("M,I,K", [(300, 192, 256), (5043, 18944, 3584), (1100, 14848, 512)])
def test_linear_swiglu(M, I, K):
    """Gate and up projections with SiLU(gate) * up in the epilogue; the last
    two shapes take the 256 x 256 tile (128 gated columns per tile), oracle on
    sampled rows."""
    import paper_2607_21599_amd as daf
    A, Wgu, _, _ = di.make_linear_case(M, 2 * I, K, seed=M + I, bias=False, residual=False)
    C = torch.full((M + 3, I), 5.0, dtype=torch.bfloat16, device="cuda")
    daf.daf_linear_swiglu(M, I, K, _dev(A), _dev(Wgu), C)
    torch.cuda.synchronize()
    rows = np.arange(M) if M <= 300 else np.union1d(
        np.random.Generator(np.random.PCG64(2)).choice(M, 20, replace=False), [0, 255, 256, M - 1])
    w = di.raw_to_f32
    Wf = w(Wgu)
    ref = dec.silu_mul(dec.linear(w(A[rows]), Wf[:I]), dec.linear(w(A[rows]), Wf[I:]))
    _close(_f(C[torch.from_numpy(rows).cuda()]), ref, f"swiglu {M}x{I}x{K}")
    assert torch.all(C[M:] == 5.0), "rows past M were written"


def test_decoder_layer_batch():
    """A ragged batch of three requests (one without important tokens, one
    without a question) in both modes; the oracle runs each request on its
    own rows (the projections are row-independent)."""
    import paper_2607_21599_amd as daf
    from oracle import get as oracle_get
    model = di.TINY_MODEL
    reqs = [(300, 16, 45), (200, 9, 0), (500, 0, 75)]  # (L_d, L_q, n)
    rng = np.random.Generator(np.random.PCG64(77))
    bits, f = di.f32_to_bf16_bits, di.raw_to_f32
    wts = di.make_layer_weights(model, 78)
    w = _weights_on_gpu(model, wts)
    ow = _oracle_weights(wts)
    cfg = daf.AttnCfg(model.hq, model.hkv, model.d, daf.DAF_BF16)
    cu_doc = np.cumsum([0] + [r[0] for r in reqs])
    cu_q = np.cumsum([0] + [r[1] for r in reqs])
    cu_imp = np.cumsum([0] + [r[2] for r in reqs])
    batch = daf.Batch(cu_doc, cu_q, cu_imp)
    xs, caches, idxs = [], [], []
    for L_d, L_q, n in reqs:
        xs.append(bits(rng.standard_normal((L_d + L_q, model.hidden), dtype=np.float32)))
        caches.append(bits(rng.standard_normal((2, L_d + L_q, model.hkv, model.d), dtype=np.float32) * 0.5))
        idxs.append(np.sort(rng.choice(L_d, n, replace=False)).astype(np.int32) if n else np.zeros(0, np.int32))
    orc, sc = oracle_get(), 1.0 / np.sqrt(model.d)
    run = lambda x, pos, attn: dec.decoder_layer(x, pos, ow, attn, model.eps, model.theta,  # noqa: E731
                                                  model.hq, model.hkv, model.d)[0]
    # DAF mode: every request's important rows, then every request's question rows
    imp_x = np.concatenate([x[i] for x, i in zip(xs, idxs)])
    q_x = np.concatenate([x[L_d:] for x, (L_d, _, _) in zip(xs, reqs)])
    imp_pos = np.concatenate(idxs)
    q_pos = np.concatenate([np.arange(L_d, L_d + L_q) for L_d, L_q, _ in reqs]).astype(np.int32)
    xa = _dev(np.concatenate([imp_x, q_x]))
    kc = _dev(np.concatenate([c[0] for c in caches]))
    vc = _dev(np.concatenate([c[1] for c in caches]))
    ws_bytes = daf.daf_decoder_layer_workspace_size(cfg, w, batch, daf.DAF_LAYER_DAF)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    daf.daf_decoder_layer(cfg, w, batch, daf.DAF_LAYER_DAF, _dev(np.concatenate(idxs)),
                          _dev(np.concatenate([imp_pos, q_pos]).astype(np.int32)), xa, kc, vc, ws, ws_bytes)
    # full mode on the same batch: every row of every request
    xf = _dev(np.concatenate(xs))
    posf = np.concatenate([np.arange(L_d + L_q) for L_d, L_q, _ in reqs]).astype(np.int32)
    ws_f = daf.daf_decoder_layer_workspace_size(cfg, w, batch, daf.DAF_LAYER_FULL)
    wsf = torch.empty(ws_f, dtype=torch.uint8, device="cuda")
    daf.daf_decoder_layer(cfg, w, batch, daf.DAF_LAYER_FULL, None, _dev(posf), xf, None, None, wsf, ws_f)
    torch.cuda.synchronize()
    got_d, got_f = _f(xa), _f(xf)
    ni = len(imp_x)
    for b, (L_d, L_q, n) in enumerate(reqs):
        rows = np.concatenate([idxs[b], np.arange(L_d, L_d + L_q)]).astype(np.int64)
        ref = run(f(xs[b][rows]), rows, dec.daf_attention(orc, idxs[b], f(caches[b][0]), f(caches[b][1]), L_d, sc))
        got = np.concatenate([got_d[cu_imp[b]:cu_imp[b + 1]], got_d[ni + cu_q[b]:ni + cu_q[b + 1]]])
        if len(rows):
            _layer_close(got, ref, f"DAF batch request {b}")
        reff = run(f(xs[b]), np.arange(L_d + L_q), dec.full_attention(orc, sc))
        t0 = cu_doc[b] + cu_q[b]
        _layer_close(got_f[t0:t0 + L_d + L_q], reff, f"full batch request {b}")
