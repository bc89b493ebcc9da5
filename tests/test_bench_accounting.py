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


def test_profile_records_used_only_for_the_same_sources_and_workload(tmp_path):
    """The bench takes kernel times and HBM bytes from a committed profile
    summary only when its record line names the workload and the SHA-256 of
    the current attention sources."""
    sha = bench.attn_source_hash()
    f = tmp_path / "summary.md"
    f.write_text("# title\n\nsome text\n"
                 f"traffic-record: workload=qwen7b_32k stage1_hbm_bytes_per_launch=123 sources_sha256={sha}\n")
    rec = bench.profile_record(str(f), "traffic-record", "qwen7b_32k")
    assert bench.record_number(rec, "stage1_hbm_bytes_per_launch") == 123.0
    assert bench.record_number(rec, "absent_key") is None
    assert bench.profile_record(str(f), "traffic-record", "qwen7b_6k") == {}
    assert bench.profile_record(str(f), "trace-record", "qwen7b_32k") == {}
    f.write_text(f"traffic-record: workload=qwen7b_32k stage1_hbm_bytes_per_launch=123 sources_sha256={'0' * 64}\n")
    assert bench.profile_record(str(f), "traffic-record", "qwen7b_32k") == {}
    assert bench.profile_record(str(tmp_path / "missing.md"), "traffic-record", "qwen7b_32k") == {}


def test_committed_profiles_match_the_sources():
    """The committed summaries were taken on the attention sources in the tree
    (otherwise the bench reports their figures as null)."""
    trace = bench.profile_record(bench.TRACE_SUMMARY, "trace-record", "qwen7b_32k")
    traffic = bench.profile_record(bench.TRAFFIC_SUMMARY, "traffic-record", "qwen7b_32k")
    for key in ("stage1_avg_us", "stage2_avg_us", "merge_avg_us", "gather_avg_us"):
        assert bench.record_number(trace, key) is not None, key
    for key in ("stage1_hbm_bytes_per_launch", "stage2_hbm_bytes_per_launch", "merge_hbm_bytes_per_launch"):
        assert bench.record_number(traffic, key) is not None, key
