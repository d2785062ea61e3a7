"""Parity of the batched matrix-core path (ts_ffn_sparse / ts_moe_sparse with
batch > 1 and bf16 weights) against the fp64 oracle, and against the
single-token path (forced with the batch_path knob).

Tolerance: relative L2 <= 1e-2 (bf16 weights, fp32 accumulation).  The
batched path splits x and Combined into bf16 high / low parts, so its gate
and up values carry about 2^-16 relative error per term; sets are compared
outside |gate|, |up| < 1e-3.  Beside the stated tolerance every output is
held to the path's own accuracy: relative L2 <= 1e-4 and every element
within its worst-case rounding bound (gpu_util)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (DEV, TIGHT_BATCH, assert_elementwise, check_ffn_output, compare_sets, ffn_inputs_to_dev,
                      list_of, moe_bound, rel_l2, to_dev)
from paper_2406_05955_amd import synth

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2406_05955_amd.binding") if torch.cuda.is_available() else None

THR = 1e-3


def check_batch(inp, ref=None, union=True):
    B, H, I = inp.shape
    ref = ref or oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    out, st = ts.ffn_sparse(x, wg, wu, wd, stats=True, union=union and B <= 64)
    torch.cuda.synchronize()
    err = rel_l2(out.cpu().numpy(), ref.y)
    assert err <= 1e-2, (B, H, I, err)
    check_ffn_output(out.cpu().numpy(), ref.y, inp.x, inp.w_gate, inp.w_up, inp.w_down_t, ref.g, ref.u,
                     batched=True, what=f"batch B={B} H={H} I={I}")
    for t in range(B):
        g, u = ref.g[t], ref.u[t]
        keep_g = np.abs(g) >= THR
        keep_a = keep_g & (np.abs(u) >= THR)
        assert compare_sets(list_of(st, "gate_idx", t, "n_gate"), g > 0, keep_g) == 0, t
        assert compare_sets(list_of(st, "active_idx", t, "n_active"), (g > 0) & (u > 0), keep_a) == 0, t
    if union and B <= 64:
        ug = (ref.g > 0).any(axis=0)
        ua = ((ref.g > 0) & (ref.u > 0)).any(axis=0)
        near = ((np.abs(ref.g) < THR) | (np.abs(ref.u) < THR)).any(axis=0)
        got = st["n_union"].cpu().tolist()
        assert abs(got[0] - int(ug.sum())) <= int(near.sum()), (got, int(ug.sum()))
        assert abs(got[1] - int(ua.sum())) <= int(near.sum()), (got, int(ua.sum()))
    return out, st, ref


@pytest.mark.parametrize("B,H,I", [(2, 512, 1000), (3, 200, 130), (8, 1024, 2048), (16, 64, 33), (17, 512, 700),
                                   (32, 1000, 1500), (33, 256, 512), (64, 512, 1024), (65, 256, 300),
                                   (130, 128, 96), (5, 8, 1), (4, 4096, 3001),
                                   (256, 128, 96), (2, 8192, 300)])  # largest batch, widest rows
def test_batch_shapes(B, H, I):
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=synth.BF16, seed=[31, B, H, I])
    check_batch(inp)


def test_batch_matches_single_token_path():
    inp = synth.make_ffn(8, 2048, 4000, gate_bias=-0.84, dtype=synth.BF16, seed=32)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    a = ts.ffn_sparse(x, wg, wu, wd)
    ts.tune_set("batch_path", 1)
    try:
        b = ts.ffn_sparse(x, wg, wu, wd)
    finally:
        ts.tune_set("batch_path", 0)
    torch.cuda.synchronize()
    assert rel_l2(a.cpu().numpy(), b.cpu().numpy().astype(np.float64)) <= 1e-4


def test_batch_hot_cold_union():
    """Skewed workload: a third of the neurons open often, the rest almost
    never; per-token sparsity ~90%, union over 16 tokens ~67%."""
    bias = synth.hot_cold_bias(3000, seed=5)
    inp = synth.make_ffn(16, 1024, 3000, gate_bias=bias, dtype=synth.BF16, seed=33)
    out, st, ref = check_batch(inp)
    ua = int(((ref.g > 0) & (ref.u > 0)).any(axis=0).sum())
    assert 0.2 * 3000 < ua < 0.45 * 3000


@pytest.mark.parametrize("B,variant", [(8, "independent"), (16, "independent"), (32, "independent"),
                                       (64, "independent"), (32, "hot_cold")])
def test_mistral_shape_batch(B, variant):
    """hidden 4096, inter 14336, bf16, drawn on the device like the
    benchmark's layers: independent tokens at 90% sparsity each (8 token
    slots: one 32-row tile per gate+up workgroup; 16, 32 and 64 slots: two
    tiles per workgroup), and the skewed hot/cold variant at batch 32; every
    output compared."""
    bias = -0.8416 if variant == "independent" else synth.hot_cold_bias(14336, seed=11)
    L = synth.make_ffn_stack_torch(1, B, 4096, 14336, gate_bias=bias, dtype=synth.BF16, seed=7, device=DEV)
    inp = synth.FFNInputs(x=L["x"][0].cpu().numpy(), w_gate=synth.tensor_to_host_array(L["w_gate"][0], synth.BF16),
                          w_up=synth.tensor_to_host_array(L["w_up"][0], synth.BF16),
                          w_down_t=synth.tensor_to_host_array(L["w_down_t"][0], synth.BF16), dtype=synth.BF16,
                          gate_bias=bias)
    check_batch(inp)


def test_batch_deterministic():
    inp = synth.make_ffn(24, 1024, 2000, gate_bias=-0.84, dtype=synth.BF16, seed=34)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    nbytes = ts.ffn_workspace_bytes(24, 1024, 2000, 1)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=DEV)
    ws.view(torch.float32)[: nbytes // 4].fill_(float("nan"))
    a = ts.ffn_sparse(x, wg, wu, wd, ws=ws)
    ws.view(torch.float32)[: nbytes // 4].fill_(float("nan"))
    b = ts.ffn_sparse(x, wg, wu, wd, ws=ws)
    torch.cuda.synchronize()
    assert torch.isfinite(a).all().item()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))


def moe_check(m):
    B, H, I, E, K = m.shape
    ref = oracle.moe(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, m.dtype, K)
    out, idx, w, st = ts.moe_sparse(to_dev(m.x), to_dev(m.w_router), to_dev(m.w_gate), to_dev(m.w_up),
                                    to_dev(m.w_down_t), K, stats=True)
    torch.cuda.synchronize()
    p = np.sort(ref.probs, axis=1)[:, ::-1]
    ties = [K < E and abs(p[t, K - 1] - p[t, K]) <= 1e-6 * p[t, K - 1] for t in range(B)]
    keep = [t for t in range(B) if not ties[t]]
    assert idx.cpu().numpy()[keep].tolist() == ref.topk_idx[keep].tolist()
    o = out.cpu().numpy()
    assert rel_l2(o[keep], ref.y[keep]) <= 1e-2
    assert rel_l2(o[keep], ref.y[keep]) <= TIGHT_BATCH
    bound = moe_bound(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, ref.topk_idx, ref.topk_w, ref.g, ref.u,
                      batched=True, tokens=keep)
    assert_elementwise(o[keep], ref.y[keep], bound[keep], f"moe batch B={B} H={H} I={I} E={E} K={K}")
    for t in keep:
        for k in range(K):
            s = t * K + k
            g, u = ref.g[t, k], ref.u[t, k]
            keep_a = (np.abs(g) >= THR) & (np.abs(u) >= THR)
            n = int(st["n_active"][s])
            assert compare_sets(st["active_idx"][s, :n].cpu().numpy(), (g > 0) & (u > 0), keep_a) == 0
    return ref, out


@pytest.mark.parametrize("B,H,I,E,K", [(16, 512, 700, 8, 2), (3, 256, 130, 4, 4), (2, 1024, 333, 1, 1),
                                       (40, 256, 200, 64, 8), (16, 4096, 2048, 8, 2), (64, 128, 64, 3, 1)])
def test_moe_batch_shapes(B, H, I, E, K):
    m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=synth.BF16, seed=[35, B, H, I, E, K])
    moe_check(m)


def test_moe_batch_overflow_groups():
    """Token slots per expert group are sized for about twice the expected
    expert load; a router that sends every token to experts 0 and 1 makes
    both take further groups (each reads its weights once per group)."""
    B, H, I, E, K = 32, 1024, 1500, 8, 2
    m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=synth.BF16, seed=36)
    m.w_router[0, 0] = synth.f32_to_bf16_bits(np.float32([10.0]))[0]  # x[:, 0] = 1: a logit bias
    m.w_router[1, 0] = synth.f32_to_bf16_bits(np.float32([9.0]))[0]
    ref, out = moe_check(m)
    assert (np.sort(ref.topk_idx, axis=1) == [0, 1]).all()
    # one group per expert with slots for the whole batch: same result up to summation order
    ts.tune_set("bx_vgroup", 1)
    try:
        out1 = ts.moe_sparse(to_dev(m.x), to_dev(m.w_router), to_dev(m.w_gate), to_dev(m.w_up),
                             to_dev(m.w_down_t), K)[0]
        torch.cuda.synchronize()
    finally:
        ts.tune_set("bx_vgroup", 0)
    assert rel_l2(out.cpu().numpy(), out1.cpu().numpy()) <= 1e-5


@pytest.mark.parametrize("B,gate_bias", [(16, -1.5548), (32, -1.5548), (64, -1.5548), (16, -0.5244)])
def test_moe_batch_mixtral_shape(B, gate_bias):
    """Mixtral shape (8 experts, hidden 4096, inter 14336, bf16) at 97%
    in-expert sparsity (b = -1.5548) and at the paper's 85% (b = -0.5244)."""
    L = synth.make_moe_stack_torch(1, B, 4096, 14336, 8, 2, gate_bias=gate_bias, dtype=synth.BF16, seed=3,
                                   device=DEV)
    h = lambda t: synth.tensor_to_host_array(t, synth.BF16)  # noqa: E731
    m = synth.MoEInputs(x=L["x"][0].cpu().numpy(), w_router=h(L["w_router"][0]), w_gate=h(L["w_gate"][0]),
                        w_up=h(L["w_up"][0]), w_down_t=h(L["w_down_t"][0]), dtype=synth.BF16, top_k=2,
                        gate_bias=gate_bias)
    ref, out = moe_check(m)
    frac = 1.0 - ((ref.g > 0) & (ref.u > 0)).mean()
    want = 0.97 if gate_bias < -1 else 0.85
    assert abs(frac - want) < 0.01, frac


@pytest.mark.parametrize("B,H,I,E,K,skew,gate", [(16, 4096, 2048, 8, 2, False, 0), (2, 512, 900, 8, 2, False, 0),
                                                 (6, 1032, 700, 8, 2, False, 0), (8, 256, 200, 64, 8, False, 0),
                                                 (16, 1024, 1500, 8, 2, True, 0), (32, 2048, 1000, 8, 2, False, 0),
                                                 (64, 1024, 700, 8, 2, True, 0), (40, 256, 200, 64, 8, False, 0),
                                                 (24, 512, 333, 4, 2, False, 3), (32, 512, 300, 8, 2, False, 1),
                                                 (16, 256, 100, 8, 2, False, 2), (64, 512, 300, 2, 2, False, 0)])
def test_moe_gathered_x_matches_dispatch_fragments(B, H, I, E, K, skew, gate):
    """The router also writes every token's x split once and the gate + up
    kernels list their group's tokens and gather their columns themselves
    (no dispatch kernel).  The operands are the dispatch kernel's fragments
    bit for bit, so the output, the routing table, the report and the dense
    comparator are the same bits either way, at 8, 16, 32 and 64 token
    slots per group and with each gate + up load shape (`gate`, the bx_gate
    knob): hidden not a multiple of 1024, 64 experts (most groups empty),
    and (skew) a router that sends every token to experts 0 and 1, which
    then take further groups."""
    m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=synth.BF16, seed=[39, B, H, I, E, K])
    if skew:
        m.w_router[0, 0] = synth.f32_to_bf16_bits(np.float32([10.0]))[0]  # x[:, 0] = 1: a logit bias
        m.w_router[1, 0] = synth.f32_to_bf16_bits(np.float32([9.0]))[0]
    args = [to_dev(m.x), to_dev(m.w_router), to_dev(m.w_gate), to_dev(m.w_up), to_dev(m.w_down_t)]

    def run(knob):
        ts.tune_set("bx_xtok", knob)
        ts.tune_set("bx_gate", gate)
        try:
            out, idx, w, st = ts.moe_sparse(*args, K, stats=True)
            dense = ts.moe_dense(*args, K)[0]
            torch.cuda.synchronize()
            return [out.clone(), idx.clone(), w.clone(), dense.clone()], {k: v.clone() for k, v in st.items()}
        finally:
            ts.tune_set("bx_xtok", 0)
            ts.tune_set("bx_gate", 0)
    ga, sa = run(0)
    fr, sf = run(1)
    for a, b in zip(ga, fr):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    for k in sa:
        if k in ("gate_idx", "active_idx"):
            cnt = sa["n_gate" if k == "gate_idx" else "n_active"]
            for r in range(cnt.numel()):
                n = int(cnt[r])
                assert torch.equal(sa[k][r, :n], sf[k][r, :n]), (k, r)
        else:
            assert torch.equal(sa[k], sf[k]), k
    if skew:
        assert (torch.sort(ga[1], dim=1).values.cpu().numpy() == [0, 1]).all()
    moe_check(m)


@pytest.mark.parametrize("B,H,I,E,K", [(16, 512, 1000, 1, 1), (32, 1024, 2048, 1, 1), (64, 256, 720, 1, 1),
                                       (20, 512, 33, 1, 1), (48, 2048, 1600, 8, 2), (64, 512, 900, 8, 2),
                                       (40, 256, 200, 64, 8)])
def test_gate_up_64_row_tiles_match_32_row_tiles(B, H, I, E, K):
    """With 16 or more token slots the gate + up kernel takes two 32-row
    tiles per workgroup; its K loop and summation order are the one-tile
    kernel's, so the output, the report and the unions are the same bits
    (inter odd, below 64 and not a multiple of 32 included; empty MoE groups
    included); the dense comparator too."""
    def run(knob):
        ts.tune_set("bx_gate", knob)
        try:
            if E == 1:
                inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=synth.BF16, seed=[37, B, H, I])
                x, wg, wu, wd = ffn_inputs_to_dev(inp)
                out, st = ts.ffn_sparse(x, wg, wu, wd, stats=True, union=True)
                dense = ts.ffn_dense(x, wg, wu, wd)
            else:
                m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=synth.BF16, seed=[38, B, H, I, E, K])
                args = [to_dev(m.x), to_dev(m.w_router), to_dev(m.w_gate), to_dev(m.w_up), to_dev(m.w_down_t)]
                out, _, _, st = ts.moe_sparse(*args, K, stats=True)
                dense = ts.moe_dense(*args, K)[0]
            torch.cuda.synchronize()
            return out.clone(), {k: v.clone() for k, v in st.items()}, dense.clone()
        finally:
            ts.tune_set("bx_gate", 0)
    o64, s64, d64 = run(0)
    o32, s32, d32 = run(3)
    assert torch.equal(o64.view(torch.int32), o32.view(torch.int32))
    assert torch.equal(d64.view(torch.int32), d32.view(torch.int32))
    for k in s64:
        if k in ("gate_idx", "active_idx"):
            cnt = s64["n_gate" if k == "gate_idx" else "n_active"]
            for r in range(cnt.numel()):
                n = int(cnt[r])
                assert torch.equal(s64[k][r, :n], s32[k][r, :n]), (k, r)
        else:
            assert torch.equal(s64[k], s32[k]), k
