"""Pins for the seeded input generator (shared by both sides of parity)."""
import numpy as np
import torch

import kvp_inputs as ki


def test_splitmix64_published_vector():
    # Reference outputs of SplitMix64 started from state 1234567.
    out = ki.raw64(1234567, np.arange(3))
    assert [int(v) for v in out] == [6457827717110365317, 3203168211198807973,
                                     9817491932198370423]


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).normal(size=100000).astype(np.float32) * 3
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0]     # ties to even
    ours = ki.round_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


def test_normal_moments_and_range():
    v = ki.normal_values(0, ki.tensor_id(ki.KIND_X), np.arange(1 << 20, dtype=np.uint64), 1.0, "fp32")
    assert abs(v.mean()) < 5e-3 and abs(v.var() - 1.0) < 5e-3
    assert np.abs(v).max() <= np.sqrt(12.0) + 1e-6
    w = ki.normal_values(0, ki.tensor_id(ki.KIND_WQ, 3), np.arange(1 << 18, dtype=np.uint64), 0.02, "bf16")
    assert abs(w.std() / 0.02 - 1) < 1e-2
    assert np.array_equal(w, ki.round_to_bf16(w))


def test_logical_indexing_is_launch_independent():
    w = ki.stage_share_prefill()
    full = ki.prefill_x(w, [1], np.arange(64))
    part = ki.prefill_x(w, [1], np.arange(16, 32))
    assert np.array_equal(full[:, 16:32], part)
    c_all = ki.cache_contents(w, ki.KIND_KCACHE, 2, b=3, length=40)
    c_pre = ki.cache_contents(w, ki.KIND_KCACHE, 2, b=3, length=10)
    assert np.array_equal(c_all[:, :10], c_pre)
    assert not np.array_equal(ki.weight(w, ki.KIND_WQ, 0), ki.weight(w, ki.KIND_WQ, 1))


def test_ragged_lengths_in_range():
    w = ki.decode_128k_ragged()
    lens = w.lengths()
    assert lens.dtype == np.int32 and len(lens) == 8
    assert lens.min() >= 65536 and lens.max() <= 131071 and lens.max() < w.kv_capacity
    assert len(set(lens.tolist())) > 1


def test_workload_maps():
    assert ki.tiny_fp32().tau == [0, 0, 2, 2]
    assert ki.stage_share_prefill().tau == [0, 1, 2, 3, 4, 4, 6, 6]
    assert ki.decode_32k().tau[:4] == [0, 0, 2, 2] and len(ki.decode_32k().producers()) == 16
    assert ki.decode_128k_ragged().tau[:8] == [0, 0, 0, 0, 4, 4, 4, 4]
