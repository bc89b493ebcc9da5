"""GPU: the allocation-free layer call against daf_layer_attn.

daf_layer_attn_noalloc takes its stage-2 workspace from the library's static
device array instead of a caller buffer. Two calls in a row, the second on a
smaller layer (the array keeps the first call's contents), each compared bit
for bit with daf_layer_attn on its own copy of the same inputs, and sampled
rows against the oracle; then a batch whose workspace exceeds the array is
refused with nothing enqueued.
"""
from __future__ import annotations

import pytest
import torch

import daf_inputs as di
from parity import assert_attn_close, assert_lse_close, oracle_request, sample_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a ROCm GPU"
    import paper_2607_21599_amd as daf
    daf.lib()
    yield
    torch.cuda.synchronize()


def _noalloc(buf):
    import paper_2607_21599_amd as daf
    t = buf.t
    daf.daf_layer_attn_noalloc(buf.cfg, buf.batch, t["idx"], t["q_imp"], t["k_imp"], t["v_imp"], t["q_q"],
                               t["k_q"], t["v_q"], t["k_cache"], t["v_cache"], t["o_imp"], t["lse_imp"],
                               t["o_q"], t["lse_q"], t["hidden"])


def _check_layer(workload: str):
    from paper_2607_21599_amd.tensors import LayerBuffers
    import paper_2607_21599_amd as daf
    batch = di.make_batch(di.workload(workload))
    s = batch.shapes[0]
    print(f"[no-alloc] {workload}", flush=True)
    a = LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, s.hq, s.hkv, s.d)
    b = LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, s.hq, s.hkv, s.d)
    assert daf.daf_layer_workspace_size(b.cfg, b.batch) <= daf.daf_layer_noalloc_max_bytes()
    a.layer()
    _noalloc(b)
    torch.cuda.synchronize()
    for k in ("o_imp", "o_q", "lse_imp", "lse_q", "hidden", "k_cache", "v_cache"):
        assert torch.equal(a[k], b[k]), f"{workload}: {k} differs from daf_layer_attn"
    rows1 = sample_rows(s.n, 40, seed=11)
    rows2 = sample_rows(s.L_q, 16, seed=12)
    ref = oracle_request(batch.request(0), rows1, rows2)
    f32 = lambda t: t.detach().float().cpu().numpy()  # noqa: E731
    assert_attn_close(f32(b["o_imp"])[rows1], ref["o_imp"], s.dtype, f"{workload} stage1")
    assert_lse_close(f32(b["lse_imp"]).T[rows1], ref["lse_imp"], s.dtype, f"{workload} lse1")
    assert_attn_close(f32(b["o_q"])[rows2], ref["o_q"], s.dtype, f"{workload} stage2")
    assert_lse_close(f32(b["lse_q"]).T[rows2], ref["lse_q"], s.dtype, f"{workload} lse2")


def test_noalloc_two_calls_second_smaller():
    _check_layer("qwen7b_32k")
    _check_layer("qwen7b_6k")


def test_noalloc_refuses_oversized_batch():
    """A question of 8192 rows needs more stage-2 workspace than the static
    array holds (one key split: 8192 x 28 bf16 partial rows, 58.7 MB): the call returns DAF_ERR_WORKSPACE and writes nothing. Every
    buffer is real and sized for the shape, so even a launch would stay in
    bounds."""
    import paper_2607_21599_amd as daf
    from paper_2607_21599_amd.tensors import LayerBuffers
    shape = di.Shape("big_q", L_d=1000, L_q=8192, n=100, hq=28, hkv=4, d=128, dtype=di.BF16, seed=5)
    batch = di.make_batch([shape])
    buf = LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, 28, 4, 128)
    assert daf.daf_layer_workspace_size(buf.cfg, buf.batch) > daf.daf_layer_noalloc_max_bytes()
    before = {k: buf[k].clone() for k in ("o_imp", "o_q", "hidden", "k_cache")}
    with pytest.raises(daf.DafError) as e:
        _noalloc(buf)
    assert e.value.status == daf.DAF_ERR_WORKSPACE
    torch.cuda.synchronize()
    for k, v in before.items():
        assert torch.equal(buf[k], v), k
