"""Device buffers for a DAF layer, held in torch tensors (device memory only).

Raw host arrays are bfloat16 bit patterns (uint16) or float32; they are moved
to the GPU unchanged. ``LayerBuffers`` owns every input, output and the
workspace of one (possibly batched) layer, laid out as include/daf.h
describes, and calls the C ABI through the binding. No arithmetic of the
method happens here.
"""
from __future__ import annotations

import numpy as np
import torch

from . import (DAF_BF16, DAF_F32, DAF_FUSE_HIDDEN, DAF_FUSE_KV, DAF_SRC_TOKENS, AttnCfg, Batch,
               daf_fuse, daf_gather_important, daf_imp_self_attn, daf_layer_attn,
               daf_layer_workspace_size, daf_position_attn, daf_qdoc_attn, daf_qdoc_workspace_size)


def to_device(raw: np.ndarray, device="cuda") -> torch.Tensor:
    raw = np.ascontiguousarray(raw)
    if raw.dtype == np.uint16:
        return torch.from_numpy(raw.view(np.int16)).to(device).view(torch.bfloat16)
    if raw.dtype in (np.float32, np.int32):
        return torch.from_numpy(raw).to(device)
    raise TypeError(f"unsupported raw dtype {raw.dtype}")


def to_host_raw(t: torch.Tensor) -> np.ndarray:
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def to_host_f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy()


INPUT_KEYS = ("idx", "q_imp", "k_imp", "v_imp", "q_q", "k_q", "v_q", "k_cache", "v_cache", "hidden")


class LayerBuffers:
    """Inputs, outputs and workspace of one DAF layer call on one device."""

    def __init__(self, arrays: dict, cu_doc, cu_q, cu_imp, hq: int, hkv: int, d: int,
                 device="cuda", softmax_scale: float = 0.0):
        dtype = DAF_BF16 if arrays["q_imp"].dtype == np.uint16 else DAF_F32
        self.cfg = AttnCfg(hq, hkv, d, dtype, softmax_scale)
        self.batch = Batch(cu_doc, cu_q, cu_imp)
        self.device = device
        self.t = {k: to_device(arrays[k], device) for k in INPUT_KEYS}
        tdt = torch.bfloat16 if dtype == DAF_BF16 else torch.float32
        n_imp, n_q = int(self.batch.cu_imp[-1]), int(self.batch.cu_q[-1])
        self.t["o_imp"] = torch.zeros((n_imp, hq, d), dtype=tdt, device=device)
        self.t["o_q"] = torch.zeros((n_q, hq, d), dtype=tdt, device=device)
        self.t["lse_imp"] = torch.zeros((hq, n_imp), dtype=torch.float32, device=device)
        self.t["lse_q"] = torch.zeros((hq, n_q), dtype=torch.float32, device=device)
        self.ws_bytes = max(daf_layer_workspace_size(self.cfg, self.batch),
                            daf_qdoc_workspace_size(self.cfg, self.batch))
        self.t["ws"] = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)
        self.elem = 2 if dtype == DAF_BF16 else 4
        self.hq, self.hkv, self.d = hq, hkv, d

    def __getitem__(self, k):
        return self.t[k]

    # -- the C ABI over these buffers ------------------------------------------
    def gather_hidden(self, dst: torch.Tensor, stream=None):
        daf_gather_important(self.batch, DAF_SRC_TOKENS, self.t["hidden"], self.hq * self.d * self.elem,
                             self.t["idx"], dst, stream)

    def fuse_kv(self, stream=None):
        t = self.t
        daf_fuse(self.cfg, self.batch, DAF_FUSE_KV, t["idx"], k_imp=t["k_imp"], v_imp=t["v_imp"],
                 k_q=t["k_q"], v_q=t["v_q"], k_cache=t["k_cache"], v_cache=t["v_cache"], stream=stream)

    def fuse_hidden(self, stream=None):
        t = self.t
        daf_fuse(self.cfg, self.batch, DAF_FUSE_HIDDEN, t["idx"], o_imp=t["o_imp"], o_q=t["o_q"],
                 hidden=t["hidden"], stream=stream)

    def stage1(self, stream=None):
        t = self.t
        daf_imp_self_attn(self.cfg, self.batch, t["q_imp"], t["k_imp"], t["v_imp"], t["o_imp"],
                          t["lse_imp"], stream)

    def stage2(self, stream=None):
        t = self.t
        daf_qdoc_attn(self.cfg, self.batch, t["q_q"], t["k_cache"], t["v_cache"], t["o_q"], t["lse_q"],
                      t["ws"], self.ws_bytes, stream)

    def layer(self, stream=None):
        t = self.t
        daf_layer_attn(self.cfg, self.batch, t["idx"], t["q_imp"], t["k_imp"], t["v_imp"], t["q_q"],
                       t["k_q"], t["v_q"], t["k_cache"], t["v_cache"], t["o_imp"], t["lse_imp"],
                       t["o_q"], t["lse_q"], t["hidden"], t["ws"], self.ws_bytes, stream)

    # -- comparison patterns of one request --------------------------------------
    def prepare_patterns(self, q_full: np.ndarray | None = None):
        """Buffers of the comparison patterns (one request): the CacheBlend
        queries (important rows, then the question rows) with their original
        positions, and, if given, queries for every token (full recompute)."""
        assert len(self.batch.cu_doc) == 2, "the comparison patterns take one request"
        t = self.t
        L_d, L_q = int(self.batch.cu_doc[1]), int(self.batch.cu_q[1])
        t["q_cb"] = torch.cat([t["q_imp"], t["q_q"]]).contiguous()
        qpos = torch.arange(L_d, L_d + L_q, dtype=torch.int32, device=self.device)
        t["pos_cb"] = torch.cat([t["idx"], qpos]).contiguous()
        t["o_cb"] = torch.zeros_like(t["q_cb"])
        t["lse_cb"] = torch.zeros((self.hq, t["q_cb"].shape[0]), dtype=torch.float32, device=self.device)
        if q_full is not None:
            t["q_full"] = to_device(q_full, self.device)
            t["o_full"] = torch.zeros_like(t["q_full"])
            t["lse_full"] = torch.zeros((self.hq, t["q_full"].shape[0]), dtype=torch.float32,
                                        device=self.device)

    def cacheblend(self, stream=None):
        """Important and question rows over the whole cache, causal by position."""
        t = self.t
        daf_position_attn(self.cfg, t["q_cb"].shape[0], t["k_cache"].shape[0], t["q_cb"], t["pos_cb"],
                          t["k_cache"], t["v_cache"], t["o_cb"], t["lse_cb"], stream)

    def full_recompute(self, stream=None):
        """Every token over its prefix of the cache (causal self-attention)."""
        t = self.t
        n = t["q_full"].shape[0]
        daf_position_attn(self.cfg, n, n, t["q_full"], None, t["k_cache"], t["v_cache"], t["o_full"],
                          t["lse_full"], stream)
