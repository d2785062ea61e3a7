"""Helpers for the GPU parity tests (host <-> device marshalling, metrics)."""
import numpy as np
import torch

from paper_2406_05955_amd import synth

DEV = "cuda:0"


def to_dev(a: np.ndarray, dtype: int | None = None) -> torch.Tensor:
    """Device copy of a host array; uint16 arrays are bf16 bit patterns."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(DEV).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def rel_l2(got, want) -> float:
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    n = np.linalg.norm(want)
    if n == 0:
        return float(np.abs(got).max()) if got.size else 0.0
    return float(np.linalg.norm(got - want) / n)


def list_of(stats, key, t, count_key):
    n = int(stats[count_key][t].item())
    return stats[key][t, :n].cpu().numpy()


def compare_sets(got: np.ndarray, want_mask: np.ndarray, keep: np.ndarray):
    """got: ascending index list from the GPU; want_mask: oracle membership
    per neuron; keep: neurons whose decision is compared.  Returns the number
    of disagreements on kept neurons (after checking the list is strictly
    ascending, in range and duplicate-free)."""
    I = want_mask.shape[0]
    assert np.all(np.diff(got) > 0), "list not strictly ascending"
    assert got.size == 0 or (got[0] >= 0 and got[-1] < I)
    gm = np.zeros(I, bool)
    gm[got] = True
    return int(np.count_nonzero((gm != want_mask) & keep))


def ffn_inputs_to_dev(inp: synth.FFNInputs):
    return (to_dev(inp.x), to_dev(inp.w_gate), to_dev(inp.w_up), to_dev(inp.w_down_t))


# ---------------------------------------------------------------------------
# Per-element error bounds.  The stated tolerance (relative L2 over the whole
# output) would pass a single output element that is off by half its value.
# Each parity check therefore also bounds every element: the GPU's gate / up
# projections differ from the oracle's by at most gu * sum_j |w_ij x_j| (fp32
# accumulation of at most n terms deep: n * 2^-24; the matrix-core path adds
# the error of representing x as two bf16 parts), which moves a neuron's
# Combined value h_i by at most dh_i = |g_i| eu_i + |u_i| eg_i + eg_i eu_i, and
# only neurons whose projections lie within that error of the positive side
# can enter; the down projection then adds at most dn * sum_i |W_down[i][j]|
# |h_i| (n * 2^-24 with n the deepest summation chain).  So
#   |y_gpu[j] - y_oracle[j]| <= sum_i |W_down[i][j]| ((1 + dn) dh_i + dn |h_i|)
# over the neurons that can enter.  The bound assumes nothing about rounding
# directions (a worst-case bound), yet a single wrong element, a dropped or
# doubled row or a wrong column exceeds it (see the tight relative-L2 bound
# checked beside it).

U32 = 2.0 ** -24
# the single-token kernels: a lane sums hidden/64 products, then 6 levels of
# wave reduction; the down sums run through at most a tile's rows, the
# reduction's per-thread rows and its tree (512 covers every launch shape)
DOWN_DEPTH = 512
# the matrix-core path: x and Combined enter as high + low bf16 parts
# (relative representation error <= 2^-17 each, 2^-16 taken)
SPLIT_REP = 2.0 ** -16
TIGHT_SINGLE = 1e-5   # relative L2, single-token kernels (fp32 and bf16 weights)
TIGHT_BATCH = 1e-4    # relative L2, matrix-core path


def gu_unit_single(H: int) -> float:
    return (H / 64.0 + 16.0) * U32


def gu_unit_batch(H: int) -> float:
    return SPLIT_REP + (H / 32.0 + 64.0) * U32


def dn_unit_single() -> float:
    return DOWN_DEPTH * U32


def dn_unit_batch() -> float:
    return SPLIT_REP + DOWN_DEPTH * U32


def host_f32(w: np.ndarray) -> np.ndarray:
    """Weights as float32 (bf16 bit patterns widened exactly)."""
    return synth.bf16_bits_to_f32(w) if w.dtype == np.uint16 else np.asarray(w, np.float32)


def abs_proj(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """sum_j |w_ij x_j| for every token and neuron: [B][I] (float64)."""
    return (np.abs(np.asarray(x, np.float32)) @ np.abs(host_f32(w)).T).astype(np.float64) * 1.001


def neuron_error(g, u, Ag, Au, gu, dn, act=0, tau=0.0):
    """Per token and neuron: the coefficient of |W_down[i][j]| in the bound
    (zero for neurons that cannot enter on either side)."""
    eg, eu = gu * Ag, gu * Au
    if act == 0:
        cand = (g > -eg) & (u > -eu)
        h = np.maximum(g, 0.0) * np.maximum(u, 0.0)
        dh = np.abs(g) * eu + np.abs(u) * eg + eg * eu
    else:
        gs = g - tau
        cand = gs > -eg
        h = np.maximum(gs, 0.0) * np.abs(u)
        dh = np.abs(gs) * eu + np.abs(u) * eg + eg * eu
    return np.where(cand, (1.0 + dn) * dh + dn * h, 0.0), np.where(cand, h, 0.0)


def down_abs(coef: np.ndarray, wd: np.ndarray) -> np.ndarray:
    """sum_i coef[t][i] |W_down[i][j]|: [B][H] (float64)."""
    return (np.asarray(coef, np.float32) @ np.abs(host_f32(wd))).astype(np.float64) * 1.001


def ffn_bound(x, wg, wu, wd, g, u, gu, dn, act=0, tau=0.0, mult=None):
    """Per-element bound of the FFN output (see above).  mult [B][I]: how
    many times each neuron is taken (given lists count repeats; the top-k
    mask takes only the kept neurons); default once."""
    coef, _ = neuron_error(g, u, abs_proj(x, wg), abs_proj(x, wu), gu, dn, act, tau)
    if mult is not None:
        coef = coef * mult
    return down_abs(coef, wd) + 1e-30


def assert_elementwise(got, want, bound, what=""):
    """Every element within its bound; the message names the worst one."""
    got = np.asarray(got, np.float64)
    err = np.abs(got - want)
    ratio = err / bound
    worst = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
    assert ratio[worst] <= 1.0, (f"{what}: element {worst} off by {err[worst]:.3e}, bound {bound[worst]:.3e} "
                                 f"(value {want[worst]:.3e})")


def check_ffn_output(got, want, x, wg, wu, wd, g, u, batched=False, act=0, tau=0.0, mult=None, what="",
                     tight=True):
    """The stated relative-L2 tolerance is checked by the caller; this adds
    the tight relative-L2 bound of the kernel family and the per-element
    bound."""
    H = x.shape[1]
    gu = gu_unit_batch(H) if batched else gu_unit_single(H)
    dn = dn_unit_batch() if batched else dn_unit_single()
    got = np.asarray(got, np.float64)
    if tight:
        err = rel_l2(got, want)
        lim = TIGHT_BATCH if batched else TIGHT_SINGLE
        assert err <= lim, f"{what}: relative L2 {err:.3e} above the tight bound {lim:.0e}"
    assert_elementwise(got, want, ffn_bound(x, wg, wu, wd, g, u, gu, dn, act, tau, mult), what)


def moe_bound(x, wr, wg, wu, wd, topk_idx, topk_w, g, u, batched=False, tokens=None):
    """Per-element bound of the MoE output: each routed expert's FFN bound
    weighted by its routing weight, plus the routing weights' own error
    (logits within gu * sum_j |W_r[e][j] x_j|, so a renormalised weight is
    within a relative 2.2 x that of its value) times that expert's sum_i
    |W_down[i][j]| h_i.  g, u: the oracle's [B][K][I] projections in rank
    order; tokens: the tokens to bound (default all)."""
    B, H = x.shape
    K = topk_idx.shape[1]
    tokens = list(range(B)) if tokens is None else list(tokens)
    gu = gu_unit_batch(H) if batched else gu_unit_single(H)
    dn = dn_unit_batch() if batched else dn_unit_single()
    Ar = abs_proj(x, wr)  # [B][E]
    out = np.zeros((B, H))
    for e in np.unique(topk_idx[tokens]):
        pairs = [(t, k) for t in tokens for k in range(K) if topk_idx[t, k] == e]
        ts_ = [t for t, _ in pairs]
        xs = x[ts_]
        gs = np.stack([g[t, k] for t, k in pairs])
        us = np.stack([u[t, k] for t, k in pairs])
        coef, h = neuron_error(gs, us, abs_proj(xs, wg[e]), abs_proj(xs, wu[e]), gu, dn)
        rw = np.array([2.2 * gu * Ar[t].max() + 16 * U32 for t in ts_])
        w = np.array([topk_w[t, k] for t, k in pairs])
        c = w[:, None] * (coef + rw[:, None] * (h + coef))
        part = down_abs(c, wd[e])
        for r, t in enumerate(ts_):
            out[t] += part[r]
    return out + 1e-30
