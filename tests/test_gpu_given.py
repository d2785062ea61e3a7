"""Parity of the given-list FFN (ts_ffn_sparse_given, the activation-predictor
interface) against the fp64 oracle's given-list function on the same seeded
inputs and lists, through the C ABI.

Tolerances: relative L2 of the output <= 1e-5 with fp32 weights and <= 1e-2
with bf16 weights (fp32 accumulation in both).  The counts (listed entries
with a positive gate / non-zero Combined activation) must match the oracle
exactly except for entries whose gate or up projection lies within the
rounding threshold (|value| < 1e-6 for fp32 weights, < 1e-4 for bf16): fp32
and fp64 may take different sides there."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, check_ffn_output, ffn_inputs_to_dev, rel_l2, to_dev
from paper_2406_05955_amd import synth

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2406_05955_amd.binding") if torch.cuda.is_available() else None


def tol_for(dtype):
    return 1e-5 if dtype == synth.F32 else 1e-2


def thr_for(dtype):
    return 1e-6 if dtype == synth.F32 else 1e-4


def random_lists(rng, B, I, maxc, with_bad=True):
    idx = rng.integers(0, I, size=(B, maxc)).astype(np.int32)
    if with_bad and maxc >= 4:
        idx[:, 0] = -5          # skipped
        idx[:, maxc // 2] = I   # skipped
        idx[:, -1] = idx[:, 1]  # repeated
    return idx


def check(inp, idx, count, stats=True):
    B, H, I = inp.shape
    ref = oracle.ffn_given(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype, idx, count)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    out, st = ts.ffn_sparse_given(x, wg, wu, wd, to_dev(idx), to_dev(np.asarray(count, np.int32)), stats=True)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    err = rel_l2(got, ref.y)
    assert err <= tol_for(inp.dtype), (B, H, I, err)
    d = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    # each listed neuron counts as often as it is listed (within count)
    mult = np.zeros((B, I))
    for t in range(B):
        n = min(max(int(count[t]), 0), idx.shape[1])
        lst = idx[t, :n]
        np.add.at(mult[t], lst[(lst >= 0) & (lst < I)], 1.0)
    check_ffn_output(got, ref.y, inp.x, inp.w_gate, inp.w_up, inp.w_down_t, d.g, d.u, mult=mult,
                     what=f"given B={B} H={H} I={I}")
    if stats:
        thr = thr_for(inp.dtype)
        for t in range(B):
            n = min(max(int(count[t]), 0), idx.shape[1])
            lst = np.array([i for i in idx[t, :n] if 0 <= i < I], np.int64)
            near_g = int((np.abs(d.g[t, lst]) < thr).sum()) if lst.size else 0
            near_u = int((np.abs(d.u[t, lst]) < thr).sum()) if lst.size else 0
            assert abs(int(st["n_gate"][t]) - int(ref.n_open[t])) <= near_g
            assert abs(int(st["n_active"][t]) - int(ref.n_active[t])) <= near_g + near_u
    return got, ref


@pytest.mark.parametrize("B,H,I,dtype,maxc", [
    (1, 512, 1792, synth.F32, 400),       # the small fp32 workload's shape
    (3, 520, 999, synth.BF16, 333),       # ragged hidden / inter / lists
    (2, 4096, 2048, synth.BF16, 1000),
    (5, 256, 300, synth.F32, 7),          # lists shorter than a chunk
    (2, 1024, 4000, synth.BF16, 4000),    # many chunks
    (256, 128, 300, synth.F32, 50),       # the largest batch
])
def test_given_random_lists(B, H, I, dtype, maxc):
    rng = np.random.default_rng(100 + B + H)
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=[41, B, H, I])
    idx = random_lists(rng, B, I, maxc)
    count = np.array([maxc - (3 * t if B < 64 else t % maxc) for t in range(B)], np.int32)
    count[-1] = maxc + 50  # clamped to max_count
    check(inp, idx, count)


def test_given_empty_and_negative_counts():
    inp = synth.make_ffn(3, 256, 500, gate_bias=0.0, dtype=synth.BF16, seed=42)
    idx = random_lists(np.random.default_rng(1), 3, 500, 64)
    got, ref = check(inp, idx, np.array([0, -7, 64], np.int32))
    assert np.all(got[0] == 0.0) and np.all(got[1] == 0.0)
    assert np.any(got[2] != 0.0)


@pytest.mark.parametrize("dtype", [synth.F32, synth.BF16])
def test_given_gate_set_equals_sparse(dtype):
    """The list G_t reported by ts_ffn_sparse gives the sparse (= dense) result;
    adding neurons outside G_t (closed gates) changes nothing beyond rounding."""
    B, H, I = 2, 1024, 3000
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=dtype, seed=43)
    d = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    sp, st = ts.ffn_sparse(x, wg, wu, wd, stats=True)
    torch.cuda.synchronize()
    ng = st["n_gate"].cpu().numpy()
    maxc = int(ng.max()) + 200
    idx = np.full((B, maxc), -1, np.int32)
    rng = np.random.default_rng(44)
    count = np.zeros(B, np.int32)
    for t in range(B):
        g = st["gate_idx"][t, :ng[t]].cpu().numpy()
        extra = rng.choice(np.setdiff1d(np.arange(I), g), size=200, replace=False).astype(np.int32)
        lst = np.concatenate([g, extra])
        rng.shuffle(lst)
        idx[t, :lst.size] = lst
        count[t] = lst.size
    got, _ = check(inp, idx, count)
    assert rel_l2(got, d.y) <= tol_for(dtype)
    # exactly G, ascending
    idx2 = np.full((B, maxc), -1, np.int32)
    for t in range(B):
        g = st["gate_idx"][t, :ng[t]].cpu().numpy()
        idx2[t, :g.size] = g
    got2, _ = check(inp, idx2, ng.astype(np.int32))
    assert rel_l2(got2, d.y) <= tol_for(dtype)
    assert rel_l2(got2, sp.cpu().numpy()) <= 1e-5


def test_given_missing_neurons_is_the_approximation():
    """Dropping half of A_t leaves exactly those terms out (parity with the
    given-list oracle) and moves the output away from the dense result."""
    B, H, I = 1, 512, 1792
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=synth.F32, seed=0)
    d = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, synth.F32)
    A = d.active_set(0)
    keep = np.concatenate([d.gate_set(0)[~np.isin(d.gate_set(0), A)], A[::2]]).astype(np.int32)
    idx = keep[None, :]
    got, ref = check(inp, idx, np.array([keep.size], np.int32))
    assert rel_l2(got, d.y) > 1e-2


@pytest.mark.parametrize("tile", [8, 32, 128])
def test_given_chunk_sizes(tile):
    inp = synth.make_ffn(2, 2048, 2500, gate_bias=-0.84, dtype=synth.BF16, seed=45)
    idx = random_lists(np.random.default_rng(tile), 2, 2500, 900)
    ts.tune_set("ffn_tile", tile)
    try:
        check(inp, idx, np.array([900, 613], np.int32))
    finally:
        ts.tune_set("ffn_tile", 0)


def test_given_mistral_shape_gate_list():
    """The Mistral-7B FFN shape (hidden 4096, inter 14336, bf16) at 90%
    sparsity with the exact gate list: parity with the oracle and with the
    sparse path."""
    inp = synth.make_ffn(1, 4096, 14336, gate_bias=-0.8416, dtype=synth.BF16, seed=46)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    sp, st = ts.ffn_sparse(x, wg, wu, wd, stats=True)
    torch.cuda.synchronize()
    n = int(st["n_gate"][0])
    idx = st["gate_idx"][:, :n].contiguous()
    cnt = torch.tensor([n], dtype=torch.int32, device=DEV)
    out = ts.ffn_sparse_given(x, wg, wu, wd, idx, cnt)
    torch.cuda.synchronize()
    ref = oracle.ffn_given(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, synth.BF16, idx.cpu().numpy(), [n])
    assert rel_l2(out.cpu().numpy(), ref.y) <= 1e-2
    assert rel_l2(out.cpu().numpy(), ref.y) <= 1e-5  # same bf16 values, fp32 accumulation
    assert rel_l2(out.cpu().numpy(), sp.cpu().numpy()) <= 1e-5


def test_given_deterministic():
    inp = synth.make_ffn(2, 1024, 2000, gate_bias=-0.5, dtype=synth.BF16, seed=47)
    idx = to_dev(random_lists(np.random.default_rng(2), 2, 2000, 700))
    cnt = torch.tensor([700, 500], dtype=torch.int32, device=DEV)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    a = ts.ffn_sparse_given(x, wg, wu, wd, idx, cnt).clone()
    b = ts.ffn_sparse_given(x, wg, wu, wd, idx, cnt)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
