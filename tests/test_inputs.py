"""The seeded input generator: bf16 rounding, determinism, shapes, FLOP count."""
import numpy as np
import pytest
import torch

from paper_2402_15627_amd import inputs as pin


def test_round_to_bf16_matches_torch_including_ties():
    r = np.random.default_rng(5)
    a = (r.standard_normal(200000) * np.exp(r.uniform(-30, 30, 200000))).astype(np.float32)
    # exact ties between two bf16 neighbours, both parities
    ties = (np.arange(1, 2001, dtype=np.uint32) << 16 | np.uint32(0x8000)).view(np.float32)
    a = np.concatenate([a, ties, -ties, np.float32([0.0, -0.0, np.inf, -np.inf])])
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(pin.round_to_bf16(a).view(np.uint32), ref.view(np.uint32))


def test_make_inputs_deterministic_and_shaped():
    s = pin.WORKLOADS["tiny_f32"]
    a = pin.make_inputs(s, seed=0)
    b = pin.make_inputs(s, seed=0)
    c = pin.make_inputs(s, seed=1)
    for n in a:
        np.testing.assert_array_equal(a[n], b[n])
        assert a[n].dtype == np.float32
    assert not np.array_equal(a["x"], c["x"])
    assert a["x"].shape == (1, 128, 256) and a["dy"].shape == (1, 128, 256)
    assert a["w_in"].shape == (s.n_in, 256) and a["w_out"].shape == (256, s.k_out)
    np.testing.assert_array_equal(a["gamma"], 1.0)  # the tiny workload fixes gamma = 1, beta = 0
    np.testing.assert_array_equal(a["beta"], 0.0)
    assert abs(a["w_in"].std() - 0.02) < 1e-3


def test_bf16_workload_values_are_bf16_exact():
    s = pin.WORKLOADS["13b_shape"].with_(seq=64, hidden=256, heads=2, ffn=512, window=16)
    a = pin.make_inputs(s, seed=0)
    for n, v in a.items():
        assert np.array_equal(pin.round_to_bf16(v), v), n


@pytest.mark.parametrize("name,flops", [
    ("tiny_f32", 6.2295e8), ("13b_shape", 3.92186e12), ("175b_tp8_share", 2.82181e12),
    ("175b_tp8_share_w512", 2.80005e12), ("long_seq_8k", 1.59451e13), ("175b_full", 2.25745e13)])
def test_model_flops(name, flops):
    assert abs(pin.model_flops(pin.WORKLOADS[name]) / flops - 1) < 1e-4


def test_visible_pairs_brute_force():
    for S in (1, 5, 17):
        for W in (1, 2, 5, 17, 40):
            brute = sum(1 for i in range(S) for j in range(S) if 0 <= i - j < W)
            assert pin.visible_pairs(S, W) == brute
