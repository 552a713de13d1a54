"""The seeded generator: shapes, counts and determinism (CPU only)."""
import numpy as np
import pytest

import synth

EXPECTED_N = {"tiny": 32, "llada": 77, "dream": 128, "long": 205, "wide": 614}


@pytest.mark.parametrize("name", list(synth.CONFIGS))
def test_shapes_and_counts(name):
    s = synth.make_step(name, 0, with_weight=False)
    c = synth.CONFIGS[name]
    LB = c["L"] * c["B"]
    assert s.q.shape == (LB, c["Hq"], c["D"]) and s.q.dtype == np.uint16
    assert s.k_lane.shape == (LB, c["Hkv"], c["D"])
    assert s.k_pre.shape == (c["P"], c["Hkv"], c["D"])
    assert s.hidden.shape == (LB, c["d"])
    assert s.N == EXPECTED_N[name]
    assert np.all(np.diff(s.row_pos) > 0) and s.is_masked.sum() == s.N
    assert np.all(s.parent < np.arange(c["L"])) and np.all(s.parent >= -1)
    if name == "wide":
        assert s.n_ref == 410 and np.all(np.diff(s.refresh_idx) > 0)
    if name == "llada":
        assert list(s.parent) == [-1, 0, 1, 2]
    # depth bound of the random trees
    for i in range(c["L"]):
        depth, j = 0, int(s.parent[i])
        while j >= 0:
            depth, j = depth + 1, int(s.parent[j])
        assert depth <= c["depth_max"]


def test_deterministic_and_bf16_roundtrip():
    a = synth.make_step("tiny", 5)
    b = synth.make_step("tiny", 5)
    assert np.array_equal(a.W, b.W) and np.array_equal(a.q, b.q)
    x = np.array([1.0, -2.5, 3.140625, 1e-3, 65504.0], np.float32)
    assert np.array_equal(synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(x))[:3], x[:3])
    # round-to-nearest-even on an exact halfway pattern
    half = np.array([0x3F808000], np.uint32).view(np.float32)
    assert synth.f32_to_bf16_bits(half)[0] == 0x3F80
    half_up = np.array([0x3F818000], np.uint32).view(np.float32)
    assert synth.f32_to_bf16_bits(half_up)[0] == 0x3F82


def test_weight_independent_of_threads():
    w1 = synth.lm_head_weight(3, 1500, 64, rows_per_chunk=256, threads=1)
    w4 = synth.lm_head_weight(3, 1500, 64, rows_per_chunk=256, threads=4)
    assert np.array_equal(w1, w4)
    f = synth.bf16_bits_to_f32(w1)
    assert abs(f.std() - 1 / 8) < 0.01
