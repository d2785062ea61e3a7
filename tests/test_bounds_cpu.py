"""The per-element error bounds the GPU parity tests apply (gpu_util), checked
on the CPU: an fp32 evaluation of the FFN and of the MoE layer (numpy float32
products and sums, a different summation order from both the kernels and the
oracle) stays inside them, and the mistakes a kernel could make do not: a
dropped active row, a doubled row, one output element off by half its value,
two output columns swapped, a routing weight off by 1%.  So the bounds are
neither too tight for correct fp32 arithmetic nor loose enough to hide a
wrong result."""
import numpy as np
import pytest

import oracle
from gpu_util import (TIGHT_SINGLE, assert_elementwise, check_ffn_output, dn_unit_single, ffn_bound,
                      gu_unit_single, host_f32, moe_bound, rel_l2)
from paper_2406_05955_amd import synth


def fp32_ffn(inp):
    x = inp.x.astype(np.float32)
    wg, wu, wd = (host_f32(w) for w in (inp.w_gate, inp.w_up, inp.w_down_t))
    g, u = x @ wg.T, x @ wu.T
    return (np.maximum(g, 0) * np.maximum(u, 0)) @ wd


@pytest.mark.parametrize("B,H,I,dtype", [(1, 512, 1792, synth.F32), (3, 1024, 3000, synth.BF16),
                                         (1, 4096, 4000, synth.BF16)])
def test_ffn_bound_passes_fp32_and_rejects_mistakes(B, H, I, dtype):
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=[91, B, H, I])
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype)
    y = fp32_ffn(inp).astype(np.float64)
    args = (inp.x, inp.w_gate, inp.w_up, inp.w_down_t, ref.g, ref.u)
    check_ffn_output(y, ref.y, *args, what="fp32")  # tight relative L2 and every element
    bound = ffn_bound(*args, gu_unit_single(H), dn_unit_single())
    assert float(np.max(np.abs(y - ref.y) / bound)) < 0.05  # far inside

    wd = host_f32(inp.w_down_t)
    act = np.nonzero((ref.g[0] > 0) & (ref.u[0] > 0))[0]
    i = int(act[len(act) // 2])
    term = ref.g[0, i] * ref.u[0, i] * wd[i].astype(np.float64)
    for name, bad in (("dropped row", -term), ("doubled row", term)):
        yb = y.copy()
        yb[0] += bad
        with pytest.raises(AssertionError):
            check_ffn_output(yb, ref.y, *args, what=name, tight=False)
        assert rel_l2(yb, ref.y) > TIGHT_SINGLE  # the tight relative L2 alone also sees it
    j = int(np.argmax(np.abs(ref.y[0])))
    yb = y.copy()
    yb[0, j] *= 1.5
    with pytest.raises(AssertionError):
        check_ffn_output(yb, ref.y, *args, what="one element", tight=False)
    yb = y.copy()
    yb[0, [j, (j + 7) % H]] = yb[0, [(j + 7) % H, j]]
    with pytest.raises(AssertionError):
        check_ffn_output(yb, ref.y, *args, what="swapped columns", tight=False)


def test_moe_bound_passes_fp32_and_rejects_a_wrong_weight():
    B, H, I, E, K = 4, 512, 700, 8, 2
    m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=synth.BF16, seed=92)
    ref = oracle.moe(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, m.dtype, K)
    x = m.x.astype(np.float32)
    y = np.zeros((B, H))
    ys = np.zeros((B, K, H))
    for t in range(B):
        for k in range(K):
            e = ref.topk_idx[t, k]
            wg, wu, wd = (host_f32(w[e]) for w in (m.w_gate, m.w_up, m.w_down_t))
            g, u = wg @ x[t], wu @ x[t]
            ys[t, k] = (np.maximum(g, 0) * np.maximum(u, 0)) @ wd
            y[t] += np.float32(ref.topk_w[t, k]) * ys[t, k]
    bound = moe_bound(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, ref.topk_idx, ref.topk_w, ref.g, ref.u)
    assert_elementwise(y, ref.y, bound, "fp32 moe")
    yb = y.copy()
    yb[1] += 0.01 * ref.topk_w[1, 0] * ys[1, 0]  # first expert's weight 1% high
    with pytest.raises(AssertionError):
        assert_elementwise(yb, ref.y, bound, "wrong weight")
