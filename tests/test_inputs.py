"""The seeded input generator (no GPU)."""
import numpy as np
import torch

import daf_inputs as di


def test_bf16_rounding_matches_torch():
    rng = np.random.Generator(np.random.PCG64(1))
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    x[:4] = [1.0 + 2**-8, 1.0 + 3 * 2**-8, -(1.0 + 2**-8), 0.0]  # ties round to even
    ours = di.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = di.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_important_counts():
    assert di.n_important(0.15, 1024) == 154
    assert di.n_important(0.15, 32768) == 4915
    assert di.n_important(0.05, 16384) == 819
    assert di.n_important(0.30, 16384) == 4915
    assert [s.n for s in di.qwen_batch8()] == [614, 1229, 1843, 2458, 3072, 3686, 4301, 4915]


def test_requests_are_seeded_and_sorted():
    s = di.tiny_f32()
    a, b = di.make_request(s), di.make_request(s)
    for k in ("idx", "q_imp", "k_cache", "hidden"):
        assert np.array_equal(a[k], b[k])
    idx = a["idx"]
    assert idx.dtype == np.int32 and len(idx) == s.n
    assert np.all(np.diff(idx) > 0) and idx[0] >= 0 and idx[-1] < s.L_d
    t = di.qwen_16k(0.05)
    r = di.make_request(di.with_seed(t, t.seed))
    assert np.all(np.diff(r["idx"]) > 0) and len(r["idx"]) == 819


def test_batch_offsets():
    shapes = di.qwen_batch8()
    assert all(32 <= s.L_q <= 256 for s in shapes)
    assert [s.L_d for s in shapes] == [4096 * (b + 1) for b in range(8)]
    assert all(sum(s.doc_lens) == s.L_d for s in shapes)
