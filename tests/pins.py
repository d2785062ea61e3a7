"""Pins for the fp64 oracle: checks against values that do not come from the
oracle itself.  Each function takes an optional ctypes library so that the
mutation tests can run the same pins against planted-bug builds of oracle.c.

Sources of truth used here:
  * a hand-worked example (tests/golden/*.json), derived on paper from
    Eq. gated-MLP and Eq. drelu of Turbo Sparse (arXiv 2406.05955);
  * exact rational arithmetic (fractions.Fraction) on tiny inputs, with the
    oracle required to sit inside the fp64 forward-error bound of a
    recursively summed dot product, |fl(s) - s| <= gamma_n * sum|terms|,
    gamma_n = n u / (1 - n u), u = 2^-53 (Higham, Accuracy and Stability of
    Numerical Algorithms, section 3.1), propagated through the ReLU products;
  * special cases that reduce to a library routine (numpy matmul, softmax);
  * exact invariants (skipping the zero Combined activations changes no bit).
"""
from __future__ import annotations

import json
import math
import os
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np

import oracle
from paper_2406_05955_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
U = 2.0 ** -53


def gamma(n: int) -> float:
    return n * U / (1.0 - n * U)


def _load_golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _f32(a):
    return np.asarray(a, dtype=np.float32)


# ----------------------------------------------------------------------------
# Hand-worked examples


def pin_ffn_handworked(lib=None):
    gd = _load_golden("ffn_handworked.json")
    r = oracle.ffn(_f32(gd["x"]), _f32(gd["w_gate"]), _f32(gd["w_up"]), _f32(gd["w_down_t"]),
                   oracle.F32, threads=1, lib=lib)
    assert np.array_equal(r.y, np.asarray(gd["out"], np.float64)), r.y
    assert np.array_equal(r.g, np.asarray(gd["gate"], np.float64)), r.g
    assert np.array_equal(r.u, np.asarray(gd["up"], np.float64)), r.u
    for t in range(2):
        assert r.gate_set(t).tolist() == gd["gate_set"][t]
        assert r.active_set(t).tolist() == gd["active_set"][t]


def _moe_golden_inputs():
    f = _load_golden("ffn_handworked.json")
    m = _load_golden("moe_handworked.json")
    wg1 = _f32(f["w_gate"])
    wu1 = _f32(f["w_up"])
    wd1 = _f32(f["w_down_t"])
    wg = np.stack([wg1, wg1, wg1])
    wu = np.stack([wu1, wu1, wu1])
    wd = np.stack([wd1, 2 * wd1, np.full_like(wd1, 100.0)])
    return _f32(m["x"]), _f32(m["w_router"]), wg, wu, wd, m


def pin_moe_handworked(lib=None):
    x, wr, wg, wu, wd, m = _moe_golden_inputs()
    r = oracle.moe(x, wr, wg, wu, wd, oracle.F32, top_k=2, threads=1, lib=lib)
    assert r.topk_idx.tolist() == m["topk_idx"], r.topk_idx
    rr = 1.0 / (1.0 + math.e)
    assert np.allclose(r.topk_w[0], [0.5, 0.5], rtol=0, atol=0), r.topk_w
    assert np.allclose(r.topk_w[1], [1 - rr, rr], rtol=4 * U, atol=0), r.topk_w
    assert np.array_equal(r.y[0], [3.0, 18.0, 6.0]), r.y
    want1 = np.array([4.0, 2.0, -3.0]) * (1.0 + rr)
    assert np.allclose(r.y[1], want1, rtol=16 * U, atol=0), (r.y[1], want1)


# ----------------------------------------------------------------------------
# Exact rational brute force


def _exact_ffn_token(x, wg, wu, wd):
    """x [H], w* [I][H] as Fractions.  Returns exact (g, u, h, y) and the
    per-element forward-error bound of a fp64 evaluation in the oracle's
    order."""
    I, H = len(wg), len(x)
    g = [sum((wg[i][j] * x[j] for j in range(H)), Fraction(0)) for i in range(I)]
    u = [sum((wu[i][j] * x[j] for j in range(H)), Fraction(0)) for i in range(I)]
    h = [g[i] * u[i] if (g[i] > 0 and u[i] > 0) else Fraction(0) for i in range(I)]
    y = [sum((wd[i][j] * h[i] for i in range(I)), Fraction(0)) for j in range(H)]
    eg = [gamma(H) * float(sum(abs(wg[i][j] * x[j]) for j in range(H))) for i in range(I)]
    eu = [gamma(H) * float(sum(abs(wu[i][j] * x[j]) for j in range(H))) for i in range(I)]
    eh = []
    for i in range(I):
        ag, au = abs(float(g[i])), abs(float(u[i]))
        # relu is 1-Lipschitz; the product adds one rounding.
        eh.append((ag + eg[i]) * eu[i] + au * eg[i] + U * (ag + eg[i]) * (au + eu[i]))
    ey = []
    for j in range(H):
        s_abs = sum(abs(float(wd[i][j])) * (abs(float(h[i])) + eh[i]) for i in range(I))
        ey.append(gamma(I) * s_abs + sum(abs(float(wd[i][j])) * eh[i] for i in range(I)))
    return g, u, h, y, ey


def _as_fractions(a, dtype):
    vals = synth.bf16_bits_to_f32(a) if dtype == synth.BF16 else np.asarray(a, np.float32)
    return [[Fraction(float(v)) for v in row] for row in np.atleast_2d(vals)]


def _within(yhat: float, y: Fraction, bound: float) -> bool:
    return float(abs(Fraction(yhat) - y)) <= 1.5 * bound + 1e-300


BRUTE_SHAPES = [(1, 1, 1), (1, 2, 5), (3, 3, 1), (2, 8, 16), (1, 5, 3), (3, 4, 7)]


def pin_ffn_bruteforce(lib=None):
    for dtype in (synth.F32, synth.BF16):
        for k, (B, H, I) in enumerate(BRUTE_SHAPES):
            for bias in (-0.3, 0.4):
                inp = synth.make_ffn(B, H, I, gate_bias=bias, dtype=dtype, seed=[17, k, dtype],
                                     bias_feature=H > 1)
                r = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, threads=1, lib=lib)
                wg, wu, wd = (_as_fractions(w, dtype) for w in (inp.w_gate, inp.w_up, inp.w_down_t))
                for t in range(B):
                    x = [Fraction(float(v)) for v in inp.x[t]]
                    g, u, h, y, ey = _exact_ffn_token(x, wg, wu, wd)
                    for j in range(H):
                        assert _within(r.y[t, j], y[j], ey[j]), (dtype, B, H, I, t, j, r.y[t, j], float(y[j]))
                    for i in range(I):
                        assert _within(r.g[t, i], g[i], gamma(H) * sum(abs(float(wg[i][j] * x[j])) for j in range(H)))
                        assert _within(r.u[t, i], u[i], gamma(H) * sum(abs(float(wu[i][j] * x[j])) for j in range(H)))


def _dec(fr: Fraction) -> Decimal:
    return Decimal(fr.numerator) / Decimal(fr.denominator)


def pin_moe_bruteforce(lib=None):
    getcontext().prec = 60
    cases = [(1, 4, 5, 1, 1), (2, 4, 6, 4, 2), (3, 3, 4, 3, 3), (2, 6, 3, 4, 1), (1, 8, 5, 2, 2)]
    for dtype in (synth.F32, synth.BF16):
        for k, (B, H, I, E, K) in enumerate(cases):
            inp = synth.make_moe(B, H, I, E, K, gate_bias=0.0, dtype=dtype, seed=[23, k, dtype])
            r = oracle.moe(inp.x, inp.w_router, inp.w_gate, inp.w_up, inp.w_down_t, dtype, K, threads=1,
                           lib=lib)
            wr = _as_fractions(inp.w_router, dtype)
            experts = [tuple(_as_fractions(w[e], dtype) for w in (inp.w_gate, inp.w_up, inp.w_down_t))
                       for e in range(E)]
            for t in range(B):
                x = [Fraction(float(v)) for v in inp.x[t]]
                logits = [sum((wr[e][j] * x[j] for j in range(H)), Fraction(0)) for e in range(E)]
                m = max(logits)
                p = [(_dec(l - m)).exp() for l in logits]
                z = sum(p)
                p = [pe / z for pe in p]
                order = sorted(range(E), key=lambda e: (-logits[e], e))
                sel = order[:K]
                # Skip tokens whose k-th and (k+1)-th logits tie within fp64 error.
                if K < E and abs(float(logits[order[K - 1]] - logits[order[K]])) < 1e-12:
                    continue
                assert r.topk_idx[t].tolist() == sel, (r.topk_idx[t], sel)
                psel = sum(p[e] for e in sel)
                w = {e: p[e] / psel for e in sel}
                for kk, e in enumerate(sel):
                    assert abs(Decimal(float(r.topk_w[t, kk])) - w[e]) <= Decimal(1e-14), (r.topk_w[t], w)
                    assert abs(Decimal(float(r.probs[t, e])) - p[e]) <= Decimal(1e-14)
                ys = {e: _exact_ffn_token(x, *experts[e]) for e in sel}
                for j in range(H):
                    want = sum(w[e] * _dec(ys[e][3][j]) for e in sorted(sel))
                    tol = sum(float(w[e]) * 1.5 * ys[e][4][j] + 1e-14 * abs(float(ys[e][3][j])) for e in sel)
                    assert abs(float(Decimal(float(r.y[t, j])) - want)) <= tol + 1e-300, (t, j, r.y[t, j], want)


# ----------------------------------------------------------------------------
# Special cases and invariants


def pin_ffn_zero_bias(lib=None):
    inp = synth.make_ffn(2, 64, 96, gate_bias=-100.0, dtype=synth.F32, seed=5)
    r = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, oracle.F32, lib=lib)
    assert np.all(r.y == 0.0)
    assert r.n_gate.tolist() == [0, 0] and r.n_active.tolist() == [0, 0]


def pin_ffn_all_active_numpy(lib=None):
    inp = synth.make_ffn(3, 48, 80, gate_bias=100.0, dtype=synth.F32, seed=6)
    inp.w_up[:, 0] = 100.0
    r = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, oracle.F32, lib=lib)
    x = inp.x.astype(np.float64)
    g = x @ inp.w_gate.astype(np.float64).T
    u = x @ inp.w_up.astype(np.float64).T
    assert np.all(g > 0) and np.all(u > 0)
    y = (g * u) @ inp.w_down_t.astype(np.float64)
    assert np.allclose(r.y, y, rtol=1e-12, atol=1e-12 * np.abs(y).max())
    assert r.n_active.tolist() == [80, 80, 80]


def pin_ffn_sets_numpy(lib=None):
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(2, 256, 700, gate_bias=-0.84, dtype=dtype, seed=7)
        r = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, lib=lib)
        up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
        x = inp.x.astype(np.float64)
        g = x @ up(inp.w_gate).astype(np.float64).T
        u = x @ up(inp.w_up).astype(np.float64).T
        assert np.allclose(r.g, g, rtol=0, atol=1e-12)
        assert np.allclose(r.u, u, rtol=0, atol=1e-12)
        ok = (np.abs(g) > 1e-9) & (np.abs(u) > 1e-9)
        assert np.array_equal(((r.g > 0) & (r.u > 0))[ok], ((g > 0) & (u > 0))[ok])
        # the active count equals the number of positive gate*up products with an open gate
        assert r.n_active.tolist() == [int(((g[t] > 0) & (u[t] > 0)).sum()) for t in range(2)]


def pin_ffn_skipzero_bitwise(lib=None):
    """Summing only the active neurons, in ascending order, reproduces every bit
    of the dense sum: the skipped terms are exact zeros."""
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(2, 128, 640, gate_bias=-0.84, dtype=dtype, seed=8)
        r = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, lib=lib)
        up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
        wd = up(inp.w_down_t).astype(np.float64)
        for t in range(2):
            y = np.zeros(128)
            for i in r.active_set(t):
                y += wd[i] * (r.g[t, i] * r.u[t, i])
            assert np.array_equal(y.view(np.uint64), r.y[t].view(np.uint64))
            assert 0 < len(r.active_set(t)) < 640


def pin_moe_special_cases(lib=None):
    # E = 1, k = 1: the MoE layer is exactly its single expert.
    m = synth.make_moe(2, 64, 100, 1, 1, gate_bias=-0.5, dtype=synth.BF16, seed=9)
    rm = oracle.moe(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, m.dtype, 1, lib=lib)
    rf = oracle.ffn(m.x, m.w_gate[0], m.w_up[0], m.w_down_t[0], m.dtype, lib=lib)
    assert np.array_equal(rm.y, rf.y)
    assert np.all(rm.topk_w == 1.0)

    # k = E: a full softmax mixture of all experts (numpy softmax and numpy sum).
    E = 4
    m = synth.make_moe(3, 32, 40, E, E, gate_bias=0.0, dtype=synth.F32, seed=10)
    rm = oracle.moe(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, m.dtype, E, lib=lib)
    x = m.x.astype(np.float64)
    logits = x @ m.w_router.astype(np.float64).T
    p = np.exp(logits - logits.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    y = np.zeros_like(x)
    for e in range(E):
        re = oracle.ffn(m.x, m.w_gate[e], m.w_up[e], m.w_down_t[e], m.dtype, lib=lib)
        y += p[:, e:e + 1] * re.y
    assert np.allclose(rm.y, y, rtol=1e-12, atol=1e-12 * np.abs(y).max())
    assert np.allclose(np.sort(rm.topk_w, axis=1), np.sort(p, axis=1), rtol=1e-12, atol=0)

    # top-2 of 8: the chosen experts are the two largest numpy logits, weights sum to 1.
    m = synth.make_moe(6, 64, 32, 8, 2, gate_bias=-1.0, dtype=synth.BF16, seed=11)
    rm = oracle.moe(m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t, m.dtype, 2, lib=lib)
    logits = m.x.astype(np.float64) @ synth.bf16_bits_to_f32(m.w_router).astype(np.float64).T
    for t in range(6):
        order = np.argsort(-logits[t], kind="stable")
        assert rm.topk_idx[t].tolist() == order[:2].tolist()
        assert abs(rm.topk_w[t].sum() - 1.0) <= 4 * U
        assert rm.topk_w[t, 0] >= rm.topk_w[t, 1]


# ----------------------------------------------------------------------------
# Given neuron lists (the activation-predictor interface)


def _given_list(rng, I, n, extra_bad=True):
    """A list of n entries: random neurons with repeats, plus (optionally)
    entries outside [0, I) that must be skipped."""
    lst = rng.integers(0, I, size=n).astype(np.int32)
    if extra_bad and n >= 3:
        lst[0] = -1
        lst[n // 2] = I
        lst[-1] = lst[1]  # a repeat
    return lst


def pin_given_bruteforce(lib=None):
    """Exact rational sums over the listed neurons (repeats counted, entries
    outside [0, I) skipped), within the fp64 forward-error bound."""
    rng = np.random.default_rng(31)
    for dtype in (synth.F32, synth.BF16):
        for k, (B, H, I) in enumerate([(1, 4, 6), (2, 8, 16), (3, 5, 9)]):
            inp = synth.make_ffn(B, H, I, gate_bias=0.2, dtype=dtype, seed=[23, k, dtype])
            maxc = I + 3
            idx = np.stack([_given_list(rng, I, maxc) for _ in range(B)])
            count = np.array([maxc - t for t in range(B)], np.int32)
            r = oracle.ffn_given(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, idx, count, threads=1, lib=lib)
            wg, wu, wd = (_as_fractions(w, dtype) for w in (inp.w_gate, inp.w_up, inp.w_down_t))
            for t in range(B):
                x = [Fraction(float(v)) for v in inp.x[t]]
                g, u, h, _, _ = _exact_ffn_token(x, wg, wu, wd)
                lst = [int(i) for i in idx[t, :count[t]] if 0 <= i < I]
                eh = []
                for i in range(I):
                    eg = gamma(H) * float(sum(abs(wg[i][j] * x[j]) for j in range(H)))
                    eu = gamma(H) * float(sum(abs(wu[i][j] * x[j]) for j in range(H)))
                    ag, au = abs(float(g[i])), abs(float(u[i]))
                    eh.append((ag + eg) * eu + au * eg + U * (ag + eg) * (au + eu))
                for j in range(H):
                    y = sum((wd[i][j] * h[i] for i in lst), Fraction(0))
                    s_abs = sum(abs(float(wd[i][j])) * (abs(float(h[i])) + eh[i]) for i in lst)
                    bound = gamma(max(len(lst), 1)) * s_abs + sum(abs(float(wd[i][j])) * eh[i] for i in lst)
                    assert _within(r.y[t, j], y, bound), (dtype, B, H, I, t, j)
                assert r.n_open[t] == sum(1 for i in lst if g[i] > 0)
                assert r.n_active[t] == sum(1 for i in lst if g[i] > 0 and u[i] > 0)


def pin_given_numpy(lib=None):
    """Random lists (repeats, out-of-range entries, ragged counts) against a
    numpy fp64 evaluation of the same sum."""
    rng = np.random.default_rng(32)
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(3, 96, 300, gate_bias=-0.3, dtype=dtype, seed=33)
        up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
        x = inp.x.astype(np.float64)
        g = x @ up(inp.w_gate).astype(np.float64).T
        u = x @ up(inp.w_up).astype(np.float64).T
        h = np.where((g > 0) & (u > 0), g * u, 0.0)
        wd = up(inp.w_down_t).astype(np.float64)
        maxc = 180
        idx = np.stack([_given_list(rng, 300, maxc) for _ in range(3)])
        count = np.array([180, 0, 77], np.int32)
        r = oracle.ffn_given(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, idx, count, lib=lib)
        for t in range(3):
            lst = np.array([i for i in idx[t, :count[t]] if 0 <= i < 300], np.int64)
            y = h[t, lst] @ wd[lst] if len(lst) else np.zeros(96)
            assert np.allclose(r.y[t], y, rtol=1e-12, atol=1e-12 * max(np.abs(y).max(), 1e-300))
            assert r.n_open[t] == int((g[t, lst] > 0).sum())
            assert r.n_active[t] == int(((g[t, lst] > 0) & (u[t, lst] > 0)).sum())
        assert np.all(r.y[1] == 0.0)


def pin_given_exact_sets_bitwise(lib=None):
    """A list holding every active neuron in ascending order (G_t, or all
    neurons) reproduces every bit of the dense oracle: the neurons it leaves
    out contribute exact zeros.  A list missing one active neuron misses
    exactly that neuron's term."""
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(2, 128, 400, gate_bias=-0.84, dtype=dtype, seed=34)
        rd = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, lib=lib)
        allrows = np.tile(np.arange(400, dtype=np.int32), (2, 1))
        r = oracle.ffn_given(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, allrows, [400, 400], lib=lib)
        assert np.array_equal(r.y.view(np.uint64), rd.y.view(np.uint64))
        assert r.n_open.tolist() == rd.n_gate.tolist() and r.n_active.tolist() == rd.n_active.tolist()
        G = [rd.gate_set(t) for t in range(2)]
        idx = np.full((2, 400), -1, np.int32)
        for t in range(2):
            idx[t, :len(G[t])] = G[t]
        r = oracle.ffn_given(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, idx, [len(G[0]), len(G[1])],
                             lib=lib)
        assert np.array_equal(r.y.view(np.uint64), rd.y.view(np.uint64))
        up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
        A0 = rd.active_set(0)
        miss = A0[len(A0) // 2]
        keep = A0[A0 != miss]
        idx = np.full((1, 400), 0, np.int32)
        idx[0, :len(keep)] = keep
        r = oracle.ffn_given(inp.x[:1], inp.w_gate, inp.w_up, inp.w_down_t, dtype, idx, [len(keep)], lib=lib)
        term = up(inp.w_down_t)[miss].astype(np.float64) * (rd.g[0, miss] * rd.u[0, miss])
        assert np.allclose(r.y[0], rd.y[0] - term, rtol=1e-12, atol=1e-12 * np.abs(rd.y[0]).max())
        assert not np.allclose(r.y[0], rd.y[0], rtol=1e-9, atol=0)


# ----------------------------------------------------------------------------
# Gate-only ReLU (ReGLU) and its shifted form


def pin_act_bruteforce(lib=None):
    """Exact rational evaluation of max(0, g - tau) * u summed over neurons,
    tau in {0, 1/4}, within the fp64 forward-error bound."""
    for dtype in (synth.F32, synth.BF16):
        for k, (B, H, I) in enumerate([(1, 4, 6), (2, 8, 16), (1, 5, 9)]):
            inp = synth.make_ffn(B, H, I, gate_bias=0.1, dtype=dtype, seed=[51, k, dtype])
            wg, wu, wd = (_as_fractions(w, dtype) for w in (inp.w_gate, inp.w_up, inp.w_down_t))
            for tau in (0.0, 0.25):
                r = oracle.ffn_act(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, oracle.ACT_RELU_GATE, tau,
                                   threads=1, lib=lib)
                ft = Fraction(tau)
                for t in range(B):
                    x = [Fraction(float(v)) for v in inp.x[t]]
                    g = [sum((wg[i][j] * x[j] for j in range(H)), Fraction(0)) for i in range(I)]
                    u = [sum((wu[i][j] * x[j] for j in range(H)), Fraction(0)) for i in range(I)]
                    h = [(g[i] - ft) * u[i] if g[i] > ft else Fraction(0) for i in range(I)]
                    eh = []
                    for i in range(I):
                        eg = gamma(H) * float(sum(abs(wg[i][j] * x[j]) for j in range(H)))
                        eu = gamma(H) * float(sum(abs(wu[i][j] * x[j]) for j in range(H)))
                        ad, au = abs(float(g[i] - ft)), abs(float(u[i]))
                        eh.append((ad + eg) * eu + au * eg + 2 * U * (ad + eg) * (au + eu))
                    for j in range(H):
                        y = sum((wd[i][j] * h[i] for i in range(I)), Fraction(0))
                        s_abs = sum(abs(float(wd[i][j])) * (abs(float(h[i])) + eh[i]) for i in range(I))
                        bound = gamma(I) * s_abs + sum(abs(float(wd[i][j])) * eh[i] for i in range(I))
                        assert _within(r.y[t, j], y, bound), (dtype, B, H, I, tau, t, j)


def pin_act_numpy(lib=None):
    """ReGLU / shifted gate against numpy fp64; the gate-only ReLU leaves the
    up branch unmasked, so the active set is the gate set (A = G)."""
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(2, 200, 500, gate_bias=-0.84, dtype=dtype, seed=52)
        up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
        x = inp.x.astype(np.float64)
        g = x @ up(inp.w_gate).astype(np.float64).T
        u = x @ up(inp.w_up).astype(np.float64).T
        wd = up(inp.w_down_t).astype(np.float64)
        for tau in (0.0, 0.3):
            r = oracle.ffn_act(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, oracle.ACT_RELU_GATE, tau, lib=lib)
            h = np.where(g > tau, (g - tau) * u, 0.0)
            y = h @ wd
            assert np.allclose(r.y, y, rtol=1e-12, atol=1e-12 * np.abs(y).max())
            for t in range(2):
                ok = np.abs(g[t] - tau) > 1e-9
                assert np.array_equal((r.g[t] > tau)[ok], (g[t] > tau)[ok])
                assert np.array_equal(r.active_set(t), r.gate_set(t))
        r = oracle.ffn_act(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, oracle.ACT_RELU_GATE, 1e6, lib=lib)
        assert np.all(r.y == 0.0)


def pin_act_drelu_is_dense_oracle(lib=None):
    """act 0 is the dReLU of or_ffn, bit for bit; a non-zero tau is rejected
    for it."""
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(2, 96, 300, gate_bias=-0.84, dtype=dtype, seed=53)
        ra = oracle.ffn_act(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, oracle.ACT_DRELU, 0.0, lib=lib)
        rd = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, lib=lib)
        assert np.array_equal(ra.y.view(np.uint64), rd.y.view(np.uint64))
        for t in range(2):
            assert np.array_equal(ra.active_set(t), rd.active_set(t))
    try:
        oracle.ffn_act(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, oracle.ACT_DRELU, 0.5, lib=lib)
    except RuntimeError:
        pass
    else:
        raise AssertionError("dReLU with a threshold accepted")


# ----------------------------------------------------------------------------
# Top-k magnitude mask (Eq. mask / sparsify-gated-MLP)


def _numpy_topk(inp, dtype, keep):
    up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
    x = inp.x.astype(np.float64)
    g = x @ up(inp.w_gate).astype(np.float64).T
    u = x @ up(inp.w_up).astype(np.float64).T
    h = np.where((g > 0) & (u > 0), g * u, 0.0)
    wd = up(inp.w_down_t).astype(np.float64)
    ys, nks = [], []
    for t in range(h.shape[0]):
        order = np.lexsort((np.arange(h.shape[1]), -np.abs(h[t])))[:keep]
        kept = np.sort(order)
        ys.append(h[t, kept] @ wd[kept] if kept.size else np.zeros(wd.shape[1]))
        nks.append(int((h[t, kept] != 0).sum()))
    return np.array(ys), np.array(nks), h


def pin_topk_numpy(lib=None):
    """The kept set and the masked sum against numpy (lexsort by |Combined|
    descending, index ascending)."""
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(3, 128, 600, gate_bias=-0.3, dtype=dtype, seed=71)
        for keep in (1, 17, 60, 250, 600, 900):
            y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, keep, lib=lib)
            yn, nkn, _ = _numpy_topk(inp, dtype, keep)
            assert np.allclose(y, yn, rtol=1e-12, atol=1e-12 * max(np.abs(yn).max(), 1e-300)), (dtype, keep)
            assert nk.tolist() == nkn.tolist()
        y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, 0, lib=lib)
        assert np.all(y == 0.0) and nk.tolist() == [0, 0, 0]


def pin_topk_keep_all_is_dense(lib=None):
    """Keeping at least every non-zero activation reproduces the dense oracle
    bit for bit (the dropped terms are exact zeros); one fewer drops exactly
    the smallest non-zero term."""
    for dtype in (synth.F32, synth.BF16):
        inp = synth.make_ffn(2, 96, 400, gate_bias=-0.84, dtype=dtype, seed=72)
        rd = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, lib=lib)
        na = int(rd.n_active.max())
        for keep in (na, 400, 10 ** 6):
            y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, dtype, keep, lib=lib)
            if keep >= na:
                assert np.array_equal(y.view(np.uint64), rd.y.view(np.uint64))
                assert nk.tolist() == rd.n_active.tolist()
        up = synth.bf16_bits_to_f32 if dtype == synth.BF16 else (lambda a: a)
        t = 0
        A = rd.active_set(t)
        hv = rd.g[t, A] * rd.u[t, A]
        small = A[np.argmin(hv)]
        y, _ = oracle.ffn_topk(inp.x[:1], inp.w_gate, inp.w_up, inp.w_down_t, dtype, len(A) - 1, lib=lib)
        term = up(inp.w_down_t)[small].astype(np.float64) * (rd.g[t, small] * rd.u[t, small])
        assert np.allclose(y[0], rd.y[0] - term, rtol=1e-12, atol=1e-12 * np.abs(rd.y[0]).max())


def pin_topk_ties_lower_index(lib=None):
    """Neurons with identical weight rows have identical Combined values; a
    cut through such a tie keeps the lower index."""
    inp = synth.make_ffn(1, 64, 50, gate_bias=0.5, dtype=synth.F32, seed=73)
    rd = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, synth.F32, lib=lib)
    A = rd.active_set(0)
    hv = rd.g[0, A] * rd.u[0, A]
    top = A[np.argmax(hv)]
    dup = [i for i in range(50) if i not in A][-1]   # an inactive neuron, becomes a copy of `top`
    lo, hi = min(top, dup), max(top, dup)
    for w in (inp.w_gate, inp.w_up):
        w[dup] = w[top]
    inp.w_down_t[dup] = synth.make_ffn(1, 64, 1, gate_bias=0.0, dtype=synth.F32, seed=74).w_down_t[0]
    y, nk = oracle.ffn_topk(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, synth.F32, 1, lib=lib)
    r = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, synth.F32, lib=lib)
    hlo = r.g[0, lo] * r.u[0, lo]
    assert r.g[0, lo] * r.u[0, lo] == r.g[0, hi] * r.u[0, hi]
    want = inp.w_down_t[lo].astype(np.float64) * hlo
    assert np.array_equal(y[0], want), (lo, hi)
    assert nk.tolist() == [1]


ALL_PINS = [pin_ffn_handworked, pin_moe_handworked, pin_ffn_bruteforce, pin_moe_bruteforce,
            pin_ffn_zero_bias, pin_ffn_all_active_numpy, pin_ffn_sets_numpy, pin_ffn_skipzero_bitwise,
            pin_moe_special_cases, pin_given_bruteforce, pin_given_numpy, pin_given_exact_sets_bitwise,
            pin_act_bruteforce, pin_act_numpy, pin_act_drelu_is_dense_oracle, pin_topk_numpy,
            pin_topk_keep_all_is_dense, pin_topk_ties_lower_index]
