"""Seeded random shapes through every single-token and batched entry point,
against the oracle with the same checks as the per-entry-point parity
tests: odd inter and hidden sizes exercise the last, shorter tiles of the
interleaved layout (tile t of T holds neurons t, t + T, ...), the batched
path's ragged unions and the MoE routing.  The draws are fixed (seed 2406),
so a failure names a reproducible case."""
import numpy as np
import pytest
import torch

import test_gpu_act
import test_gpu_ffn
import test_gpu_given
import test_gpu_moe
import test_gpu_topk
from paper_2406_05955_amd import synth

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2406_05955_amd.binding") if torch.cuda.is_available() else None

_rng = np.random.default_rng(2406)


def _shape(max_b, max_h, max_i, dtype):
    B = int(_rng.integers(1, max_b + 1))
    H = int(_rng.integers(1, max_h // 8 + 1)) * 8
    if dtype == synth.F32:
        H = min(H, 4096)
    I = int(_rng.integers(1, max_i + 1))
    return B, H, I


FFN_CASES = []
for k in range(12):
    dt = (synth.F32, synth.BF16)[k % 2]
    B, H, I = _shape(6, 2048, 5000, dt)
    FFN_CASES.append((dt, B, H, I, float(_rng.choice([-0.84, -0.3, -1.5])), k % 3 == 2))
ACT_CASES = []
for k in range(4):
    dt = (synth.F32, synth.BF16)[k % 2]
    B, H, I = _shape(4, 1024, 3000, dt)
    ACT_CASES.append((dt, B, H, I, float(_rng.uniform(0.0, 0.5))))
TOPK_CASES = []
for k in range(4):
    dt = (synth.F32, synth.BF16)[k % 2]
    B, H, I = _shape(4, 1024, 3000, dt)
    TOPK_CASES.append((dt, B, H, max(I, 64), float(_rng.uniform(0.05, 0.9))))
GIVEN_CASES = []
for k in range(4):
    dt = (synth.F32, synth.BF16)[k % 2]
    B, H, I = _shape(4, 1024, 3000, dt)
    GIVEN_CASES.append((dt, B, H, I, int(_rng.integers(1, I + 40))))
MOE_CASES = []
for k in range(4):
    dt = (synth.F32, synth.BF16)[k % 2]
    B, H, I = _shape(20, 512, 800, dt)
    E = int(_rng.integers(1, 9))
    MOE_CASES.append((dt, B, H, I, E, int(_rng.integers(1, min(E, 4) + 1))))


@pytest.mark.parametrize("dtype,B,H,I,bias,fused", FFN_CASES)
def test_random_ffn(dtype, B, H, I, bias, fused):
    inp = synth.make_ffn(B, H, I, gate_bias=bias, dtype=dtype, seed=[2406, B, H, I])
    ts.tune_set("ffn_path", 2 if fused else 0)
    try:
        test_gpu_ffn.check_ffn(inp)
    finally:
        ts.tune_set("ffn_path", 0)


@pytest.mark.parametrize("dtype,B,H,I,tau", ACT_CASES)
def test_random_act(dtype, B, H, I, tau):
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=[2407, B, H, I])
    test_gpu_act.check(inp, tau)


@pytest.mark.parametrize("dtype,B,H,I,frac", TOPK_CASES)
def test_random_topk(dtype, B, H, I, frac):
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=[2408, B, H, I])
    test_gpu_topk.check(inp, frac)


@pytest.mark.parametrize("dtype,B,H,I,maxc", GIVEN_CASES)
def test_random_given(dtype, B, H, I, maxc):
    rng = np.random.default_rng([2409, B, H, I])
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=[2409, B, H, I])
    idx = test_gpu_given.random_lists(rng, B, I, maxc)
    count = rng.integers(-2, maxc + 3, size=B).astype(np.int32)
    test_gpu_given.check(inp, idx, count)


@pytest.mark.parametrize("dtype,B,H,I,E,K", MOE_CASES)
def test_random_moe(dtype, B, H, I, E, K):
    m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=dtype, seed=[2410, B, H, I, E, K])
    test_gpu_moe.check_moe(m)
