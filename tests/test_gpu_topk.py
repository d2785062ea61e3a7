"""Parity of the top-k magnitude mask (ts_ffn_sparse_topk) against the fp64
oracle's or_ffn_topk, through the C ABI.

The kept set is decided on fp32 Combined values on the GPU and on fp64 ones
in the oracle, so each case takes `keep` where the oracle's sorted Combined
values have a clear gap between the keep-th and the next (relative 1e-4,
some hundred times the fp32 accumulation error of a projection): there both
sides keep the same neurons, and
the reported active set must equal the oracle's kept set exactly.  Outputs:
relative L2 <= 1e-5 with fp32 weights, <= 1e-2 with bf16 weights.  A call
without the report takes the other kernel sequence (the down workgroups
select for themselves); it must give the same bits as the call with it."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import check_ffn_output, compare_sets, ffn_inputs_to_dev, list_of, rel_l2
from paper_2406_05955_amd import synth

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2406_05955_amd.binding") if torch.cuda.is_available() else None


def combined(ref, t):
    return np.maximum(ref.g[t], 0.0) * np.maximum(ref.u[t], 0.0)


def clear_keep(c, want, gap):
    """The keep nearest `want` whose cut between the keep-th largest Combined
    value and the next has relative gap >= `gap`."""
    s = np.sort(c[c > 0])[::-1]
    for d in range(0, s.size):
        for k in (want - d, want + d):
            if 1 <= k < s.size and s[k - 1] - s[k] >= gap * s[k - 1]:
                return k
    raise AssertionError("no clear cut")


def kept_mask(c, keep):
    order = np.lexsort((np.arange(c.size), -c))  # descending value, then ascending index
    m = np.zeros(c.size, bool)
    m[order[:keep]] = True
    return m & (c > 0)


def check(inp, frac):
    B, H, I = inp.shape
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    gap = 1e-4
    # one keep for all tokens: it must give a clear cut on every token
    want = max(1, int(frac * np.count_nonzero(combined(ref, 0))))
    keep = clear_keep(combined(ref, 0), want, gap)
    for t in range(1, B):
        c = np.sort(combined(ref, t)[combined(ref, t) > 0])[::-1]
        if keep < c.size and c[keep - 1] - c[keep] < gap * c[keep - 1]:
            pytest.skip("no keep with a clear cut on every token for this seed")
    y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype, keep)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    out, st = ts.ffn_sparse_topk(x, wg, wu, wd, keep, stats=True)
    fast = ts.ffn_sparse_topk(x, wg, wu, wd, keep)  # no report: the down workgroups select for themselves
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), fast.view(torch.int32))
    err = rel_l2(out.cpu().numpy(), y)
    assert err <= (1e-5 if inp.dtype == synth.F32 else 1e-2), (B, H, I, keep, err)
    mult = np.stack([kept_mask(combined(ref, t), keep) for t in range(B)]).astype(np.float64)
    check_ffn_output(out.cpu().numpy(), y, inp.x, inp.w_gate, inp.w_up, inp.w_down_t, ref.g, ref.u, mult=mult,
                     what=f"topk B={B} H={H} I={I} keep={keep}")
    thr = 1e-6 if inp.dtype == synth.F32 else 1e-4
    for t in range(B):
        c = combined(ref, t)
        want_k = kept_mask(c, keep)
        near = np.abs(ref.g[t]) < thr
        # neurons whose activity the two sides may decide differently (a
        # gate, or an open gate's up, in the rounding band): when keep
        # reaches into them, the kept sets may differ by those neurons alone
        near_a = near | ((ref.g[t] > 0) & (np.abs(ref.u[t]) < thr))
        assert int(st["n_active"][t]) == int(nk[t])
        if near_a.any():
            assert abs(int(nk[t]) - np.count_nonzero(want_k)) <= np.count_nonzero(near_a)
            assert compare_sets(list_of(st, "active_idx", t, "n_active"), want_k, ~near_a) == 0
        else:
            assert int(nk[t]) == np.count_nonzero(want_k)
            assert compare_sets(list_of(st, "active_idx", t, "n_active"), want_k, np.ones(I, bool)) == 0
        assert compare_sets(list_of(st, "gate_idx", t, "n_gate"), ref.g[t] > 0, ~near) == 0
    return out, ref, keep


@pytest.mark.parametrize("B,H,I,dtype,frac", [
    (1, 512, 1792, synth.F32, 0.5),     # the small fp32 workload's shape
    (1, 512, 1792, synth.F32, 0.1),
    (3, 520, 999, synth.BF16, 0.5),     # ragged, several tokens
    (2, 4096, 2048, synth.F32, 0.3),    # fp32 rows of 1024 chunks
    (4, 2048, 3000, synth.BF16, 0.7),
    (256, 128, 200, synth.BF16, 0.5),   # the largest batch
])
def test_topk_shapes(B, H, I, dtype, frac):
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=[71, B, H, I])
    check(inp, frac)


def test_topk_mistral_shape():
    """Mistral-7B's FFN (4096 x 14336, bf16), keeping half of the active set."""
    inp = synth.make_ffn(1, 4096, 14336, gate_bias=-0.8416, dtype=synth.BF16, seed=72)
    check(inp, 0.5)


def test_topk_largest_inter():
    """inter = 16384, the largest the on-chip selection holds."""
    inp = synth.make_ffn(1, 1024, 16384, gate_bias=-0.5, dtype=synth.BF16, seed=73)
    check(inp, 0.6)


def test_topk_keep_all_and_zero():
    """keep >= |A| keeps every active neuron (the sparse FFN's result);
    keep = 0 gives zeros with the gate set still reported."""
    inp = synth.make_ffn(2, 1024, 2000, gate_bias=-0.84, dtype=synth.F32, seed=74)
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    for keep in (2000, 5000, int(ref.n_active.max())):
        out, st = ts.ffn_sparse_topk(x, wg, wu, wd, keep, stats=True)
        fast = ts.ffn_sparse_topk(x, wg, wu, wd, keep)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), fast.view(torch.int32))
        assert rel_l2(out.cpu().numpy(), ref.y) <= 1e-5
        assert np.array_equal(st["n_active"].cpu().numpy(), ref.n_active)
    out, st = ts.ffn_sparse_topk(x, wg, wu, wd, 0, stats=True)
    fast = ts.ffn_sparse_topk(x, wg, wu, wd, 0)
    torch.cuda.synchronize()
    assert not out.any().item() and not fast.any().item()
    assert not st["n_active"].any().item()
    assert np.array_equal(st["n_gate"].cpu().numpy(), ref.n_gate)


def test_topk_ties_take_lower_index():
    """Rows duplicated across the neuron axis give bitwise-equal Combined
    values on the GPU; a cut through such a pair keeps the lower index."""
    H, I = 1024, 2048
    inp = synth.make_ffn(1, H, I, gate_bias=-0.3, dtype=synth.BF16, seed=75)
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    c = combined(ref, 0)
    order = np.argsort(-c, kind="stable")
    # copy neuron a (ranked 100th) into neurons b1 < b2 above it in index,
    # in different tiles, so three neurons share one value
    a = int(order[99])
    b1, b2 = (a + 700) % I, (a + 1500) % I
    for w in (inp.w_gate, inp.w_up):
        w[b1] = w[a]
        w[b2] = w[a]
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    c = combined(ref, 0)
    v = c[a]
    above = int(np.count_nonzero(c > v))
    trio = sorted((a, b1, b2))
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    for take in (1, 2):
        keep = above + take
        y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype, keep)
        out, st = ts.ffn_sparse_topk(x, wg, wu, wd, keep, stats=True)
        fast = ts.ffn_sparse_topk(x, wg, wu, wd, keep)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), fast.view(torch.int32)), take
        got = set(list_of(st, "active_idx", 0, "n_active").tolist())
        assert set(trio[:take]) <= got and not (set(trio[take:]) & got), (take, trio)
        assert rel_l2(out.cpu().numpy(), y) <= 1e-2
        assert rel_l2(out.cpu().numpy(), y) <= 1e-5  # exact bf16 weights, fp32 accumulation
        assert int(st["n_active"][0]) == int(nk[0]) == keep


def test_topk_deterministic():
    inp = synth.make_ffn(3, 2048, 5000, gate_bias=-0.84, dtype=synth.BF16, seed=76)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    a = ts.ffn_sparse_topk(x, wg, wu, wd, 300).clone()
    b = ts.ffn_sparse_topk(x, wg, wu, wd, 300)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def test_topk_split_gate_up_kernel():
    """The gate+up kernel of the split path (rows too wide for the pipelined
    kernel take it) feeding the same selection, forced by the path knob."""
    inp = synth.make_ffn(2, 1024, 3000, gate_bias=-0.84, dtype=synth.BF16, seed=77)
    ts.tune_set("ffn_path", 1)
    try:
        check(inp, 0.4)
    finally:
        ts.tune_set("ffn_path", 0)


def test_topk_token_with_no_open_gate():
    """A token whose gates are all closed (x = e_0 meets the negative bias
    column) keeps nothing and gets a zero output; its neighbours are served
    as usual."""
    inp = synth.make_ffn(3, 1024, 2000, gate_bias=-0.84, dtype=synth.BF16, seed=78)
    inp.x[1] = 0.0
    inp.x[1, 0] = 1.0
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    assert int(ref.n_gate[1]) == 0
    keep = clear_keep(combined(ref, 0), 60, 1e-4)
    y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype, keep)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    out, st = ts.ffn_sparse_topk(x, wg, wu, wd, keep, stats=True)
    fast = ts.ffn_sparse_topk(x, wg, wu, wd, keep)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), fast.view(torch.int32))
    o = out.cpu().numpy()
    assert not o[1].any()
    assert int(st["n_gate"][1]) == 0 and int(st["n_active"][1]) == 0
    assert rel_l2(o[0], y[0]) <= 1e-2
    assert rel_l2(o[0], y[0]) <= 1e-5
    assert int(st["n_active"][0]) == int(nk[0]) == keep


def test_topk_mistral_batch64():
    """64 tokens at the Mistral shape (128-neuron tiles of the pipelined
    kernel, 14336 list positions per token): outputs and kept counts for
    every token against the oracle (a keep with a clear cut on token 0;
    other tokens compared by output only where their cut is clear)."""
    inp = synth.make_ffn(64, 4096, 14336, gate_bias=-0.8416, dtype=synth.BF16, seed=79)
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    keep = clear_keep(combined(ref, 0), 700, 1e-4)
    y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype, keep)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    out, st = ts.ffn_sparse_topk(x, wg, wu, wd, keep, stats=True)
    fast = ts.ffn_sparse_topk(x, wg, wu, wd, keep)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), fast.view(torch.int32))
    o = out.cpu().numpy()
    checked = 0
    for t in range(64):
        c = np.sort(combined(ref, t)[combined(ref, t) > 0])[::-1]
        if keep < c.size and c[keep - 1] - c[keep] < 1e-4 * c[keep - 1]:
            continue  # no clear cut on this token: GPU and oracle may keep different neurons
        assert int(st["n_active"][t]) == int(nk[t]), t
        assert rel_l2(o[t], y[t]) <= 1e-2, t
        assert rel_l2(o[t], y[t]) <= 1e-5, t
        checked += 1
    assert checked >= 48
