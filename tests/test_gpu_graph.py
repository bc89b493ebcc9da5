"""GPU: the hot path captured into a HIP graph and replayed.

The library's calls enqueue kernels and stream/event operations only (no
allocation, no copy, no memset, no synchronisation), so a caller can capture a
layer's attention into a graph; the layer call's second stream joins the
capture through its fork event and rejoins it through its join event. Each test
captures once and replays several times. Between the replays the program
restores the inputs it changes in place (hidden rows, the KV cache), scrambles
every output with its own eager kernels and synchronises; every replay must
then reproduce the eager result bit for bit (the kernels are deterministic).
If a kernel escaped the capture (ran once while capturing instead of on every
replay), its outputs would stay scrambled and the comparison fails.
"""
from __future__ import annotations

import pytest
import torch

import daf_inputs as di

pytestmark = pytest.mark.gpu

OUTS = ("o_imp", "lse_imp", "o_q", "lse_q", "hidden", "k_cache", "v_cache")
REPLAYS = 4


def _shape(name, L_d, L_q, n, seed):
    return di.Shape(name, L_d=L_d, L_q=L_q, n=n, hq=28, hkv=4, d=128, dtype=di.BF16, seed=seed)


CASES = {
    "qwen7b_6k": lambda: di.workload("qwen7b_6k"),
    "ragged_batch": lambda: [_shape("r0", 3000, 77, 450, 81), _shape("r1", 700, 128, 700, 82),
                             _shape("r2", 5000, 5, 40, 83)],
}


class _Run:
    def __init__(self, shapes):
        from paper_2607_21599_amd.tensors import LayerBuffers
        batch = di.make_batch(shapes)
        s = batch.shapes[0]
        self.buf = LayerBuffers(batch.arrays, batch.cu_doc, batch.cu_q, batch.cu_imp, s.hq, s.hkv, s.d)
        self.gath = torch.empty((int(batch.cu_imp[-1]), s.hq * s.d), dtype=self.buf["hidden"].dtype, device="cuda")
        self.initial = {k: self.buf[k].clone() for k in ("hidden", "k_cache", "v_cache")}

    def reset(self):
        """Eager work between replays: inputs changed in place back to their
        initial values, every output scrambled."""
        for k, v in self.initial.items():
            self.buf[k].copy_(v)
        for k in ("o_imp", "o_q"):
            self.buf[k].fill_(-7.0)
        for k in ("lse_imp", "lse_q"):
            self.buf[k].fill_(float("nan"))
        self.gath.fill_(3.0)
        torch.cuda.synchronize()

    def snapshot(self):
        return {**{k: self.buf[k].clone() for k in OUTS}, "gathered": self.gath.clone()}

    def check(self, ref, what):
        got = self.snapshot()
        for k, v in ref.items():
            assert torch.equal(got[k].view(torch.uint8), v.view(torch.uint8)), f"{what}: {k} differs from eager"


def _replay_and_check(run: _Run, fn, what):
    # eager reference; the first call also creates the layer call's second stream
    run.reset()
    fn()
    torch.cuda.synchronize()
    run.reset()
    fn()
    torch.cuda.synchronize()
    ref = run.snapshot()
    run.reset()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    for i in range(REPLAYS):
        run.reset()
        g.replay()
        torch.cuda.synchronize()
        run.check(ref, f"{what} replay {i}")
    del g
    torch.cuda.synchronize()


@pytest.mark.parametrize("case", list(CASES))
def test_layer_call_graph(case):
    """gather + daf_layer_attn (two streams inside) captured as one graph."""
    run = _Run(CASES[case]())

    def step():
        run.buf.gather_hidden(run.gath)
        run.buf.layer()

    _replay_and_check(run, step, f"{case} layer call")


@pytest.mark.parametrize("case", list(CASES))
def test_stage_calls_graph(case):
    """The separate entry points (KV write-back, stage 1, stage 2 with its
    merge, hidden fusion) captured in order as one graph."""
    run = _Run(CASES[case]())

    def steps():
        b = run.buf
        b.gather_hidden(run.gath)
        b.fuse_kv()
        b.stage1()
        b.stage2()
        b.fuse_hidden()

    _replay_and_check(run, steps, f"{case} stage calls")
