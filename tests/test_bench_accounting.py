"""CPU: the benchmark's algorithmic work counts, which every reported rate
and roofline fraction divides by.

FLOP: each visible (query, key) pair of one head costs 2·D for the score and
2·D for its share of P·V. The visible pairs are counted here by brute force
from explicit masks (stage 1: the condensed sequence's lower triangle; stage 2:
question row j over cache rows 0 .. L_d + j), independently of the closed
forms the benchmark uses. Bytes: every operand read once and every output
written once, spelled out per tensor at the benchmark's 32k shape.
"""
from __future__ import annotations

import numpy as np
import pytest

import bench
import daf_inputs as di


def _pairs_stage1(n: int) -> int:
    return int(np.tril(np.ones((n, n), dtype=bool)).sum())


def _pairs_stage2(L_d: int, L_q: int) -> int:
    keys = np.arange(L_d + L_q)[None, :]
    rows = np.arange(L_q)[:, None]
    return int((keys <= L_d + rows).sum())


@pytest.mark.parametrize("L_d,L_q,n,hq,hkv,d", [(300, 17, 45, 28, 4, 128), (1000, 64, 150, 8, 2, 64),
                                                (64, 1, 64, 28, 4, 128), (0, 5, 0, 14, 2, 128)])
def test_flop_counts_match_brute_force_masks(L_d, L_q, n, hq, hkv, d):
    s = di.Shape("acct", L_d=L_d, L_q=L_q, n=n, hq=hq, hkv=hkv, d=d, dtype=di.BF16, seed=1)
    w = bench.work([s])
    assert w["stage1_flop"] == 4 * d * hq * _pairs_stage1(n)
    assert w["stage2_flop"] == 4 * d * hq * _pairs_stage2(L_d, L_q)


def test_flop_counts_add_over_a_batch():
    shapes = di.workload("qwen7b_batch8")
    total = bench.work(shapes)
    parts = [bench.work([s]) for s in shapes]
    for k in total:
        assert total[k] == sum(p[k] for p in parts), k


def test_bytes_at_32k():
    w = bench.work(di.workload("qwen7b_32k"))
    n, L_d, L_q = 4915, 32768, 128
    q_row, kv_row = 28 * 128 * 2, 4 * 128 * 2  # bf16 bytes per token row of Q/O and of K or V
    # stage 1: q_imp read, o_imp written, k_imp and v_imp read
    assert w["stage1_bytes"] == n * q_row * 2 + n * kv_row * 2 == 80_527_360
    # stage 2: the whole [L_d + L_q] cache's K and V read, q_q read, o_q written
    assert w["stage2_bytes"] == (L_d + L_q) * kv_row * 2 + L_q * q_row * 2 == 69_206_016
    # gather: n hidden rows read and written; hidden fusion: n + L_q rows read and written;
    # KV write-back: n + L_q rows of K and of V read and written
    assert w["gather_bytes"] == 2 * n * q_row
    assert w["fuse_hidden_bytes"] == 2 * (n + L_q) * q_row
    assert w["fuse_kv_bytes"] == 2 * (n + L_q) * 2 * kv_row
