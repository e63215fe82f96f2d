"""The seeded input generator: bf16 rounding and reproducibility."""
import numpy as np
import torch

from lora_synth import CONFIGS, Shape, bf16_bits_to_f32, gen_inputs, gen_ternary_inputs, round_to_bf16_bits


def test_round_ties_to_even():
    x = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 1 + 2 ** -8 + 2 ** -20], np.float32)
    got = bf16_bits_to_f32(round_to_bf16_bits(x))
    assert got.tolist() == [1.0, 1.0, 1 + 2 ** -6, -1.0, 1 + 2 ** -7]


def test_round_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    ours = round_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_seeded_and_shaped():
    s = CONFIGS["tiny"][0]
    assert (s.m, s.n, s.k, s.r, s.alpha, s.seed) == (256, 512, 512, 8, 16.0, 0)
    a, b = gen_inputs(s), gen_inputs(s)
    for key in a:
        assert np.array_equal(a[key], b[key])
    assert a["X"].shape == (256, 512) and a["W"].shape == (512, 512)
    assert a["A"].shape == (8, 512) and a["B"].shape == (512, 8) and a["dY"].shape == (256, 512)
    assert all(v.dtype == np.uint16 for v in a.values())
    seeds = [p.seed for p in CONFIGS["llama2_13b_layer"]]
    assert seeds == [4000 + i for i in range(7)]


def test_distributions():
    s = Shape("d", 512, 1024, 2048, 16, 32.0, 5)
    t = {k: bf16_bits_to_f32(v).astype(np.float64) for k, v in gen_inputs(s).items()}
    assert abs(t["X"].std() - 1) < 0.01 and abs(t["dY"].std() - 1) < 0.01
    assert abs(t["W"].std() * np.sqrt(2048) - 1) < 0.01
    assert np.abs(t["A"]).max() <= 1 / np.sqrt(2048) * (1 + 2 ** -8)
    assert abs(t["B"].std() - 0.02) < 0.001


def test_ternary_values():
    t = gen_ternary_inputs(64, 96, 128, 8, 3)
    for v in t.values():
        assert set(np.unique(bf16_bits_to_f32(v)).tolist()) <= {-1.0, 0.0, 1.0}
