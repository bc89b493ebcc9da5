"""Python binding of the DAF C ABI (``libdaf.so``, declared in include/daf.h).

Argument marshalling only: every step of the DAF layer runs in the HIP
kernels of ``libdaf.so``. Tensor arguments may be torch tensors on the GPU
(their data pointers are passed) or plain integer device addresses. Streams
default to torch's current stream. Nothing here falls back to a CPU path: if
the library is not built, every call raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

__all__ = [
    "DAF_OK", "DAF_BF16", "DAF_F32", "DAF_SRC_TOKENS", "DAF_SRC_DOCS", "DAF_FUSE_KV",
    "DAF_FUSE_HIDDEN", "DafError", "AttnCfg", "Batch", "lib", "library_path",
    "daf_gather_important", "daf_imp_self_attn", "daf_position_attn", "daf_qdoc_workspace_size", "daf_qdoc_attn",
    "daf_fuse", "daf_layer_workspace_size", "daf_layer_attn", "daf_layer_noalloc_max_bytes",
    "daf_layer_attn_noalloc", "daf_check_indices", "daf_select_important",
    "daf_linear", "daf_linear_swiglu", "daf_rmsnorm", "daf_rope", "daf_silu_mul", "daf_decoder_layer_workspace_size",
    "daf_decoder_layer", "LayerWeights", "DAF_LAYER_DAF", "DAF_LAYER_FULL",
    "daf_status_string", "daf_last_error", "daf_version", "EXPORTED",
]

DAF_OK = 0
DAF_ERR_INVALID_ARG, DAF_ERR_ALIGNMENT, DAF_ERR_UNSUPPORTED, DAF_ERR_WORKSPACE, DAF_ERR_HIP = 1, 2, 3, 4, 5
DAF_BF16, DAF_F32 = 0, 1
DAF_SRC_TOKENS, DAF_SRC_DOCS = 0, 1
DAF_FUSE_KV, DAF_FUSE_HIDDEN = 1, 2
DAF_LAYER_DAF, DAF_LAYER_FULL = 0, 1

# every symbol include/daf.h declares
EXPORTED = [
    "daf_gather_important", "daf_imp_self_attn", "daf_position_attn", "daf_qdoc_workspace_size", "daf_qdoc_attn",
    "daf_fuse", "daf_layer_workspace_size", "daf_layer_attn", "daf_layer_noalloc_max_bytes",
    "daf_layer_attn_noalloc", "daf_check_indices", "daf_select_important",
    "daf_linear", "daf_linear_swiglu", "daf_rmsnorm", "daf_rope", "daf_silu_mul", "daf_decoder_layer_workspace_size",
    "daf_decoder_layer", "daf_status_string", "daf_last_error", "daf_version",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_PKG, "libdaf.so")


class DafError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{_status_name(status)}: {detail}")
        self.status = status
        self.detail = detail


class AttnCfg(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float)]

    def __init__(self, n_q_heads, n_kv_heads, head_dim, dtype=DAF_BF16, softmax_scale=0.0):
        super().__init__(n_q_heads, n_kv_heads, head_dim, dtype, softmax_scale)


class _BatchC(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("cu_doc", ctypes.POINTER(ctypes.c_int32)),
                ("cu_q", ctypes.POINTER(ctypes.c_int32)), ("cu_imp", ctypes.POINTER(ctypes.c_int32))]


class Batch:
    """Host prefix arrays of a ragged batch, kept alive with their C struct."""

    def __init__(self, cu_doc, cu_q, cu_imp):
        self.cu_doc = np.ascontiguousarray(cu_doc, dtype=np.int32)
        self.cu_q = np.ascontiguousarray(cu_q, dtype=np.int32)
        self.cu_imp = np.ascontiguousarray(cu_imp, dtype=np.int32)
        p = ctypes.POINTER(ctypes.c_int32)
        self.c = _BatchC(len(self.cu_doc) - 1, self.cu_doc.ctypes.data_as(p),
                         self.cu_q.ctypes.data_as(p), self.cu_imp.ctypes.data_as(p))

    @classmethod
    def single(cls, L_d: int, L_q: int, n: int) -> "Batch":
        return cls([0, L_d], [0, L_q], [0, n])


_vp = ctypes.c_void_p


class LayerWeights(ctypes.Structure):
    """daf_layer_weights_t: device pointers of one decoder layer's weights.
    Build it with ``from_tensors``, which keeps the tensors alive."""
    _fields_ = [("w_in", _vp), ("wq", _vp), ("bq", _vp), ("wk", _vp), ("bk", _vp), ("wv", _vp), ("bv", _vp),
                ("wo", _vp), ("w_post", _vp), ("wgu", _vp), ("wd", _vp), ("hidden", ctypes.c_int32),
                ("inter", ctypes.c_int32), ("eps", ctypes.c_float), ("rope_theta", ctypes.c_float)]

    @classmethod
    def from_tensors(cls, t: dict, hidden: int, inter: int, eps: float, rope_theta: float) -> "LayerWeights":
        names = ["w_in", "wq", "bq", "wk", "bk", "wv", "bv", "wo", "w_post", "wgu", "wd"]
        w = cls(*[t[n].data_ptr() for n in names], hidden, inter, eps, rope_theta)
        w._keep = t
        return w


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded libdaf.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(library_path):
            raise RuntimeError(f"{library_path} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(library_path)
        cfgp, bp = ctypes.POINTER(AttnCfg), ctypes.POINTER(_BatchC)
        i32, i64, u32, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_size_t
        sig = {
            "daf_gather_important": (i32, [bp, i32, _vp, i64, _vp, _vp, _vp]),
            "daf_imp_self_attn": (i32, [cfgp, bp, _vp, _vp, _vp, _vp, _vp, _vp]),
            "daf_position_attn": (i32, [cfgp, ctypes.c_int32, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp, _vp,
                                        _vp]),
            "daf_select_important": (i32, [cfgp, bp, ctypes.c_int32, _vp, _vp, _vp, _vp, _vp]),
            "daf_qdoc_workspace_size": (sz, [cfgp, bp]),
            "daf_qdoc_attn": (i32, [cfgp, bp, _vp, _vp, _vp, _vp, _vp, _vp, sz, _vp]),
            "daf_fuse": (i32, [cfgp, bp, u32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
            "daf_layer_workspace_size": (sz, [cfgp, bp]),
            "daf_layer_attn": (i32, [cfgp, bp, _vp] + [_vp] * 13 + [_vp, sz, _vp]),
            "daf_layer_noalloc_max_bytes": (sz, []),
            "daf_layer_attn_noalloc": (i32, [cfgp, bp, _vp] + [_vp] * 13 + [_vp]),
            "daf_check_indices": (i32, [bp, _vp, _vp, _vp]),
            "daf_linear": (i32, [i64, i32, i32, _vp, _vp, _vp, _vp, _vp, _vp]),
            "daf_linear_swiglu": (i32, [i64, i32, i32, _vp, _vp, _vp, _vp]),
            "daf_rmsnorm": (i32, [i64, i32, _vp, _vp, ctypes.c_float, _vp, _vp]),
            "daf_rope": (i32, [i64, i32, i32, i64, _vp, _vp, ctypes.c_float, _vp]),
            "daf_silu_mul": (i32, [i64, i32, _vp, _vp, _vp]),
            "daf_decoder_layer_workspace_size": (sz, [cfgp, ctypes.POINTER(LayerWeights), bp, i32]),
            "daf_decoder_layer": (i32, [cfgp, ctypes.POINTER(LayerWeights), bp, i32, _vp, _vp, _vp, _vp, _vp,
                                        _vp, sz, _vp]),
            "daf_status_string": (ctypes.c_char_p, [i32]),
            "daf_last_error": (ctypes.c_char_p, []),
            "daf_version": (i32, []),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def _status_name(status: int) -> str:
    try:
        return lib().daf_status_string(status).decode()
    except Exception:  # noqa: BLE001 - only used to format an error message
        return f"status {status}"


def _ptr(x):
    """Device address of a tensor (or an int address, or None)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x or None
    return x.data_ptr() or None


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream


def _check(status: int):
    if status != DAF_OK:
        raise DafError(status, lib().daf_last_error().decode())


def _cfgp(cfg: AttnCfg):
    return ctypes.byref(cfg)


def _bp(batch: Batch):
    return ctypes.byref(batch.c)


# ---- the C ABI, one function per entry point --------------------------------
def daf_gather_important(batch: Batch, src_layout: int, src, row_bytes: int, idx, dst, stream=None):
    _check(lib().daf_gather_important(_bp(batch), src_layout, _ptr(src), row_bytes, _ptr(idx),
                                      _ptr(dst), _stream(stream)))


def daf_imp_self_attn(cfg: AttnCfg, batch: Batch, q_imp, k_imp, v_imp, o_imp, lse_imp=None,
                      stream=None):
    _check(lib().daf_imp_self_attn(_cfgp(cfg), _bp(batch), _ptr(q_imp), _ptr(k_imp), _ptr(v_imp),
                                   _ptr(o_imp), _ptr(lse_imp), _stream(stream)))


def daf_position_attn(cfg: AttnCfg, n_rows: int, n_keys: int, q, q_pos, k, v, o, lse=None, stream=None):
    _check(lib().daf_position_attn(_cfgp(cfg), n_rows, n_keys, _ptr(q), _ptr(q_pos), _ptr(k), _ptr(v),
                                   _ptr(o), _ptr(lse), _stream(stream)))


def daf_linear(M: int, N: int, K: int, A, W, bias, residual, C, stream=None):
    _check(lib().daf_linear(M, N, K, _ptr(A), _ptr(W), _ptr(bias), _ptr(residual), _ptr(C), _stream(stream)))


def daf_linear_swiglu(M: int, I: int, K: int, A, Wgu, C, stream=None):
    _check(lib().daf_linear_swiglu(M, I, K, _ptr(A), _ptr(Wgu), _ptr(C), _stream(stream)))


def daf_rmsnorm(rows: int, width: int, x, w, eps: float, y, stream=None):
    _check(lib().daf_rmsnorm(rows, width, _ptr(x), _ptr(w), eps, _ptr(y), _stream(stream)))


def daf_rope(rows: int, n_heads: int, head_dim: int, row_stride: int, x, pos, theta: float, stream=None):
    _check(lib().daf_rope(rows, n_heads, head_dim, row_stride, _ptr(x), _ptr(pos), theta, _stream(stream)))


def daf_silu_mul(rows: int, width: int, gu, out, stream=None):
    _check(lib().daf_silu_mul(rows, width, _ptr(gu), _ptr(out), _stream(stream)))


def daf_decoder_layer_workspace_size(cfg: AttnCfg, w: LayerWeights, batch: Batch, mode: int) -> int:
    return int(lib().daf_decoder_layer_workspace_size(_cfgp(cfg), ctypes.byref(w), ctypes.byref(batch.c), mode))


def daf_decoder_layer(cfg: AttnCfg, w: LayerWeights, batch: Batch, mode: int, idx, pos, x, k_cache, v_cache,
                      workspace, ws_bytes: int, stream=None):
    _check(lib().daf_decoder_layer(_cfgp(cfg), ctypes.byref(w), ctypes.byref(batch.c), mode, _ptr(idx), _ptr(pos),
                                   _ptr(x), _ptr(k_cache), _ptr(v_cache), _ptr(workspace), ws_bytes,
                                   _stream(stream)))


def daf_select_important(cfg: AttnCfg, batch: Batch, k_fresh, k_cached, scores, idx, stream=None):
    """k_fresh / k_cached: sequences (one entry per selection layer) of device
    tensors or addresses, passed as host arrays of device pointers."""
    nl = len(k_fresh)
    fresh = (ctypes.c_void_p * max(nl, 1))(*[_ptr(t) for t in k_fresh])
    cached = (ctypes.c_void_p * max(len(k_cached), 1))(*[_ptr(t) for t in k_cached])
    _check(lib().daf_select_important(_cfgp(cfg), _bp(batch), nl, ctypes.cast(fresh, ctypes.c_void_p),
                                      ctypes.cast(cached, ctypes.c_void_p), _ptr(scores), _ptr(idx),
                                      _stream(stream)))


def daf_qdoc_workspace_size(cfg: AttnCfg, batch: Batch) -> int:
    return int(lib().daf_qdoc_workspace_size(_cfgp(cfg), _bp(batch)))


def daf_qdoc_attn(cfg: AttnCfg, batch: Batch, q_q, k_cache, v_cache, o_q, lse_q, workspace,
                  ws_bytes: int, stream=None):
    _check(lib().daf_qdoc_attn(_cfgp(cfg), _bp(batch), _ptr(q_q), _ptr(k_cache), _ptr(v_cache),
                               _ptr(o_q), _ptr(lse_q), _ptr(workspace), ws_bytes, _stream(stream)))


def daf_fuse(cfg: AttnCfg, batch: Batch, flags: int, idx, k_imp=None, v_imp=None, k_q=None,
             v_q=None, k_cache=None, v_cache=None, o_imp=None, o_q=None, hidden=None, stream=None):
    _check(lib().daf_fuse(_cfgp(cfg), _bp(batch), flags, _ptr(idx), _ptr(k_imp), _ptr(v_imp),
                          _ptr(k_q), _ptr(v_q), _ptr(k_cache), _ptr(v_cache), _ptr(o_imp), _ptr(o_q),
                          _ptr(hidden), _stream(stream)))


def daf_layer_workspace_size(cfg: AttnCfg, batch: Batch) -> int:
    return int(lib().daf_layer_workspace_size(_cfgp(cfg), _bp(batch)))


def daf_layer_attn(cfg: AttnCfg, batch: Batch, idx, q_imp, k_imp, v_imp, q_q, k_q, v_q, k_cache,
                   v_cache, o_imp, lse_imp, o_q, lse_q, hidden, workspace, ws_bytes: int,
                   stream=None):
    _check(lib().daf_layer_attn(_cfgp(cfg), _bp(batch), _ptr(idx), _ptr(q_imp), _ptr(k_imp),
                                _ptr(v_imp), _ptr(q_q), _ptr(k_q), _ptr(v_q), _ptr(k_cache),
                                _ptr(v_cache), _ptr(o_imp), _ptr(lse_imp), _ptr(o_q), _ptr(lse_q),
                                _ptr(hidden), _ptr(workspace), ws_bytes, _stream(stream)))


def daf_layer_noalloc_max_bytes() -> int:
    return int(lib().daf_layer_noalloc_max_bytes())


def daf_layer_attn_noalloc(cfg: AttnCfg, batch: Batch, idx, q_imp, k_imp, v_imp, q_q, k_q, v_q, k_cache,
                           v_cache, o_imp, lse_imp, o_q, lse_q, hidden, stream=None):
    _check(lib().daf_layer_attn_noalloc(_cfgp(cfg), _bp(batch), _ptr(idx), _ptr(q_imp), _ptr(k_imp),
                                        _ptr(v_imp), _ptr(q_q), _ptr(k_q), _ptr(v_q), _ptr(k_cache),
                                        _ptr(v_cache), _ptr(o_imp), _ptr(lse_imp), _ptr(o_q), _ptr(lse_q),
                                        _ptr(hidden), _stream(stream)))


def daf_check_indices(batch: Batch, idx, d_bad_count, stream=None):
    _check(lib().daf_check_indices(_bp(batch), _ptr(idx), _ptr(d_bad_count), _stream(stream)))


def daf_status_string(status: int) -> str:
    return lib().daf_status_string(status).decode()


def daf_last_error() -> str:
    return lib().daf_last_error().decode()


def daf_version() -> int:
    return int(lib().daf_version())
