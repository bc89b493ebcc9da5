"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects bad arguments before touching the GPU."""
import ctypes
import os
import re

import pytest

import paper_2607_21599_amd as daf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "daf.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(daf_[a-z_]+)\s*\(", text)))


def test_header_symbols_exported():
    names = _declared()
    assert len(names) >= 11
    assert sorted(daf.EXPORTED) == names
    lib = ctypes.CDLL(daf.library_path)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    assert daf.daf_status_string(0) == "DAF_OK"
    assert daf.daf_status_string(5) == "DAF_ERR_HIP"
    assert daf.daf_version() >= 100


FAKE = 0x10000  # an aligned non-null address; never dereferenced on these paths


def _cfg(**kw):
    a = dict(n_q_heads=28, n_kv_heads=4, head_dim=128, dtype=daf.DAF_BF16, softmax_scale=0.0)
    a.update(kw)
    return daf.AttnCfg(**a)


@pytest.mark.parametrize("cfg,status", [
    (dict(n_kv_heads=3), daf.DAF_ERR_INVALID_ARG),
    (dict(n_q_heads=0), daf.DAF_ERR_INVALID_ARG),
    (dict(head_dim=96), daf.DAF_ERR_UNSUPPORTED),
    (dict(dtype=7), daf.DAF_ERR_UNSUPPORTED),
    (dict(softmax_scale=-1.0), daf.DAF_ERR_INVALID_ARG),
    (dict(softmax_scale=float("nan")), daf.DAF_ERR_INVALID_ARG),
])
def test_bad_cfg(cfg, status):
    b = daf.Batch.single(100, 8, 10)
    with pytest.raises(daf.DafError) as e:
        daf.daf_imp_self_attn(_cfg(**cfg), b, FAKE, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == status
    assert daf.daf_last_error()


def test_bad_batches():
    c = _cfg()
    with pytest.raises(daf.DafError) as e:  # n > L_d
        daf.daf_imp_self_attn(c, daf.Batch.single(10, 4, 11), FAKE, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # decreasing prefix
        daf.daf_imp_self_attn(c, daf.Batch([0, 10, 5], [0, 1, 2], [0, 1, 2]), FAKE, FAKE, FAKE, FAKE,
                              None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # a decrease whose int32 difference would wrap to positive
        daf.daf_imp_self_attn(c, daf.Batch([0, 2_000_000_000, -2_000_000_000], [0, 1, 2], [0, 1, 2]), FAKE, FAKE,
                              FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # prefix not starting at 0
        daf.daf_imp_self_attn(c, daf.Batch([1, 10], [0, 1], [0, 1]), FAKE, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG


def test_pointer_checks():
    c = _cfg()
    b = daf.Batch.single(100, 8, 10)
    with pytest.raises(daf.DafError) as e:
        daf.daf_imp_self_attn(c, b, FAKE + 8, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_ALIGNMENT
    with pytest.raises(daf.DafError) as e:
        daf.daf_imp_self_attn(c, b, None, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:
        daf.daf_gather_important(b, daf.DAF_SRC_TOKENS, FAKE, 24, FAKE, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_ALIGNMENT
    with pytest.raises(daf.DafError) as e:
        daf.daf_gather_important(b, 5, FAKE, 32, FAKE, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:
        daf.daf_fuse(c, b, 0, FAKE, stream=0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # KV mode without the caches
        daf.daf_fuse(c, b, daf.DAF_FUSE_KV, FAKE, k_imp=FAKE, v_imp=FAKE, k_q=FAKE, v_q=FAKE, stream=0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG


def test_workspace_checks():
    c = _cfg()
    b = daf.Batch.single(32768, 128, 4915)
    need = daf.daf_qdoc_workspace_size(c, b)
    assert need == daf.daf_layer_workspace_size(c, b)
    # 128 rows x 18 splits x 28 heads: 128 bf16 partial outputs and one fp32 LSE,
    # each region 256-byte aligned
    assert need == 128 * 18 * 28 * 128 * 2 + ((128 * 18 * 28 * 4 + 255) // 256) * 256
    # a 32-row question: 7 (head, 32-row) units per KV head in 2 workgroups,
    # 8 workgroups per split over 513 key tiles; about 512 workgroups of equal
    # share give splits of 9 tiles, so 57 splits
    b32 = daf.Batch.single(32768, 32, 4915)
    assert daf.daf_qdoc_workspace_size(c, b32) == 32 * 57 * 28 * 128 * 2 + ((32 * 57 * 28 * 4 + 255) // 256) * 256
    for ws, nbytes, status in [(None, need, daf.DAF_ERR_WORKSPACE), (FAKE, need - 1, daf.DAF_ERR_WORKSPACE),
                               (FAKE + 4, need, daf.DAF_ERR_ALIGNMENT)]:
        with pytest.raises(daf.DafError) as e:
            daf.daf_qdoc_attn(c, b, FAKE, FAKE, FAKE, FAKE, None, ws, nbytes, 0)
        assert e.value.status == status
    assert daf.daf_qdoc_workspace_size(_cfg(head_dim=96), b) == 0
    assert daf.daf_qdoc_workspace_size(c, daf.Batch.single(100, 0, 3)) == 0


def test_empty_work_is_a_no_op():
    c = _cfg()
    b = daf.Batch.single(0, 0, 0)
    daf.daf_imp_self_attn(c, b, None, None, None, None, None, 0)
    daf.daf_qdoc_attn(c, b, None, None, None, None, None, None, 0, 0)
    daf.daf_layer_attn(c, b, *([None] * 14), None, 0, 0)
    daf.daf_gather_important(b, daf.DAF_SRC_TOKENS, None, 16, None, None, 0)


def test_position_attn_checks():
    c = _cfg()
    with pytest.raises(daf.DafError) as e:  # negative sizes
        daf.daf_position_attn(c, -1, 10, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # bottom-right causal needs n_rows <= n_keys
        daf.daf_position_attn(c, 11, 10, FAKE, None, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # positions without keys
        daf.daf_position_attn(c, 3, 0, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:
        daf.daf_position_attn(c, 3, 10, FAKE, FAKE + 2, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_ALIGNMENT
    with pytest.raises(daf.DafError) as e:
        daf.daf_position_attn(c, 3, 10, FAKE, FAKE, None, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # K/V of one call must fit 32-bit byte offsets
        daf.daf_position_attn(c, 3, 1 << 22, FAKE, FAKE, FAKE, FAKE, FAKE, None, 0)
    assert e.value.status == daf.DAF_ERR_UNSUPPORTED
    daf.daf_position_attn(c, 0, 10, None, None, None, None, None, None, 0)  # no rows: no-op


def test_select_important_checks():
    c = _cfg()
    b = daf.Batch.single(100, 8, 10)
    with pytest.raises(daf.DafError) as e:  # no layers
        daf.daf_select_important(c, b, [], [], FAKE, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # more than 8 layers
        daf.daf_select_important(c, b, [FAKE] * 9, [FAKE] * 9, FAKE, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:
        daf.daf_select_important(c, b, [FAKE, FAKE + 4], [FAKE, FAKE], FAKE, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_ALIGNMENT
    with pytest.raises(daf.DafError) as e:
        daf.daf_select_important(c, b, [FAKE], [FAKE], None, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_INVALID_ARG
    with pytest.raises(daf.DafError) as e:  # token rows wider than 4 KiB
        daf.daf_select_important(_cfg(n_q_heads=32, n_kv_heads=16, dtype=daf.DAF_F32), b, [FAKE], [FAKE],
                                 FAKE, FAKE, 0)
    assert e.value.status == daf.DAF_ERR_UNSUPPORTED
    daf.daf_select_important(c, daf.Batch.single(0, 3, 0), [FAKE], [FAKE], None, None, 0)  # no documents


def _weights(**kw):
    a = dict(hidden=256, inter=512, eps=1e-6, rope_theta=1e6)
    a.update(kw)
    return daf.LayerWeights(*([FAKE] * 11), a["hidden"], a["inter"], a["eps"], a["rope_theta"])


def _status(fn, *args):
    with pytest.raises(daf.DafError) as e:
        fn(*args)
    return e.value.status


def test_linear_and_row_op_checks():
    assert _status(daf.daf_linear, 10, 100, 64, FAKE, FAKE, None, None, FAKE, 0) == daf.DAF_ERR_UNSUPPORTED
    assert _status(daf.daf_linear, 10, 128, 96, FAKE, FAKE, None, None, FAKE, 0) == daf.DAF_ERR_UNSUPPORTED
    assert _status(daf.daf_linear, -1, 128, 64, FAKE, FAKE, None, None, FAKE, 0) == daf.DAF_ERR_INVALID_ARG
    assert _status(daf.daf_linear, 10, 128, 64, None, FAKE, None, None, FAKE, 0) == daf.DAF_ERR_INVALID_ARG
    assert _status(daf.daf_linear, 10, 128, 64, FAKE, FAKE, FAKE + 2, None, FAKE, 0) == daf.DAF_ERR_ALIGNMENT
    daf.daf_linear(0, 128, 64, None, None, None, None, None, 0)  # no rows: nothing to do
    assert _status(daf.daf_linear_swiglu, 10, 96, 64, FAKE, FAKE, FAKE, 0) == daf.DAF_ERR_UNSUPPORTED
    assert _status(daf.daf_linear_swiglu, 10, 128, 100, FAKE, FAKE, FAKE, 0) == daf.DAF_ERR_UNSUPPORTED
    assert _status(daf.daf_linear_swiglu, 10, 128, 64, FAKE, None, FAKE, 0) == daf.DAF_ERR_INVALID_ARG
    daf.daf_linear_swiglu(0, 128, 64, None, None, None, 0)
    assert _status(daf.daf_rmsnorm, 4, 12, FAKE, FAKE, 1e-6, FAKE, 0) == daf.DAF_ERR_UNSUPPORTED
    assert _status(daf.daf_rmsnorm, 4, 16, FAKE, FAKE, -1.0, FAKE, 0) == daf.DAF_ERR_INVALID_ARG
    daf.daf_rmsnorm(0, 16, None, None, 1e-6, None, 0)
    assert _status(daf.daf_rope, 4, 2, 63, 128, FAKE, FAKE, 1e4, 0) == daf.DAF_ERR_INVALID_ARG
    assert _status(daf.daf_rope, 4, 2, 64, 100, FAKE, FAKE, 1e4, 0) == daf.DAF_ERR_INVALID_ARG
    assert _status(daf.daf_rope, 4, 2, 64, 128, FAKE, FAKE, 0.0, 0) == daf.DAF_ERR_INVALID_ARG
    assert _status(daf.daf_rope, 4, 2, 64, 128, FAKE, FAKE + 2, 1e4, 0) == daf.DAF_ERR_ALIGNMENT
    assert _status(daf.daf_silu_mul, 4, 12, FAKE, FAKE, 0) == daf.DAF_ERR_UNSUPPORTED


def test_decoder_layer_checks():
    c = _cfg(n_q_heads=4, n_kv_heads=2, head_dim=64)
    b = daf.Batch.single(600, 32, 90)
    w = _weights()
    L = daf.daf_decoder_layer
    ws = daf.daf_decoder_layer_workspace_size(c, w, b, daf.DAF_LAYER_DAF)
    assert ws > 0 and daf.daf_decoder_layer_workspace_size(c, w, b, 7) == 0
    full = daf.daf_decoder_layer_workspace_size(c, w, b, daf.DAF_LAYER_FULL)
    assert full > ws  # every token recomputed
    args = (daf.DAF_LAYER_DAF, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, ws, 0)
    assert _status(L, _cfg(n_q_heads=4, n_kv_heads=2, head_dim=64, dtype=daf.DAF_F32), w, b, *args) == \
        daf.DAF_ERR_UNSUPPORTED
    assert _status(L, c, _weights(hidden=200), b, *args) == daf.DAF_ERR_UNSUPPORTED
    bad = _weights()
    bad.wo = None
    assert _status(L, c, bad, b, *args) == daf.DAF_ERR_INVALID_ARG
    assert _status(L, c, w, b, 5, *args[1:]) == daf.DAF_ERR_INVALID_ARG
    assert _status(L, c, w, b, *args[:-2], ws - 1, 0) == daf.DAF_ERR_WORKSPACE
    assert _status(L, c, w, b, daf.DAF_LAYER_DAF, FAKE, None, FAKE, FAKE, FAKE, FAKE, ws, 0) == \
        daf.DAF_ERR_INVALID_ARG  # no positions
    # the full layer needs no cache or indices
    assert _status(L, c, w, b, daf.DAF_LAYER_FULL, None, FAKE, FAKE, None, None, FAKE, full - 1, 0) == \
        daf.DAF_ERR_WORKSPACE
    L(c, w, daf.Batch.single(0, 0, 0), daf.DAF_LAYER_DAF, None, None, None, None, None, None, 0, 0)  # no rows
