"""The seeded input generator: bf16 rounding and the sparsity calibration."""
from statistics import NormalDist

import numpy as np
import pytest
import torch

from paper_2406_05955_amd import synth


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38, 1e-40, 1.00390625, 1.01171875,
                                  np.inf, -np.inf], np.float32)])
    ours = synth.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(synth.bf16_bits_to_f32(ours), torch.from_numpy(a).to(torch.bfloat16).float().numpy())


@pytest.mark.parametrize("b", [-0.84, -1.5548, 0.0])
def test_gate_fraction_calibration(b):
    """Fraction of open gates over 64 seeds within 4 sigma of E_x[Phi(b / sigma_x)],
    sigma_x^2 = |x[1:]|^2 / H; combined fraction within 4 sigma of half of it."""
    H, I, n = 512, 1792, 64
    opened, active, expect = 0, 0, 0.0
    for s in range(n):
        inp = synth.make_ffn(1, H, I, gate_bias=b, dtype=synth.F32, seed=s)
        x = inp.x[0].astype(np.float64)
        g = inp.w_gate.astype(np.float64) @ x
        u = inp.w_up.astype(np.float64) @ x
        opened += int((g > 0).sum())
        active += int(((g > 0) & (u > 0)).sum())
        sig = np.sqrt((x[1:] ** 2).sum() / H)
        expect += NormalDist().cdf(b / sig)
    p = expect / n
    N = n * I
    assert abs(opened / N - p) <= 4 * np.sqrt(p * (1 - p) / N)
    q = p / 2
    assert abs(active / N - q) <= 4 * np.sqrt(q * (1 - q) / N) + 0.002


def test_bias_for_sparsity():
    assert synth.gate_bias_for_combined_sparsity(0.9) == pytest.approx(-0.8416, abs=1e-4)
    assert synth.gate_bias_for_combined_sparsity(0.99) == pytest.approx(-2.0537, abs=1e-4)
    assert synth.gate_bias_for_combined_sparsity(0.75) == pytest.approx(0.0, abs=1e-12)
    assert synth.gate_bias_for_combined_sparsity(0.5) == 8.0
    assert synth.gate_bias_for_gate_fraction(0.06) == pytest.approx(-1.5548, abs=1e-4)


def test_generator_is_seeded():
    a = synth.make_ffn(2, 64, 32, dtype=synth.BF16, seed=3)
    b = synth.make_ffn(2, 64, 32, dtype=synth.BF16, seed=3)
    for n in ("x", "w_gate", "w_up", "w_down_t"):
        assert np.array_equal(getattr(a, n), getattr(b, n))
    assert np.all(a.x[:, 0] == 1.0)
    assert np.all(synth.bf16_bits_to_f32(a.w_gate[:, 0]) == synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(
        np.float32([-0.84]))))
