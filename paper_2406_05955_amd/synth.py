"""Seeded synthetic inputs for the sparse dReLU FFN and its MoE form.

This module only draws and lays out inputs; it performs none of the FFN's
arithmetic.  Both the HIP path and the CPU oracle consume what it returns.

Workload recipe (the paper's trained weights are not available; these
synthetic layers have the real Mistral-7B / Mixtral FFN shapes, H=4096 and
I=14336, and the per-layer sparsity levels reported in the paper's section 6.2):

* x ~ N(0, 1) per token, with x[:, 0] = 1 so that column 0 of W_gate acts as
  a gate bias (the paper's FFN has no bias, section 3.2 footnote; the bias
  column is the generator's knob for sparsity, not part of the method).
* W_gate, W_up, W_down_t ~ N(0, 1/H), all stored neuron-major [I][H]; row i of
  W_down_t is neuron i's output row (the paper's W_down row i, Eq. gated-MLP).
* W_gate[i][0] = b for every neuron i.  Then P(gate_i > 0) = Phi(b) and, since
  the up projection is symmetric, P(Combined_i != 0) = Phi(b) / 2.
* MoE: router W_r [E][H] ~ N(0, 1/H) is drawn first, then every expert's
  three matrices; experts are packed [E][I][H].

Small layers use numpy's PCG64 (``default_rng``), drawn in float64 and
rounded to float32.  Large stacks (hundreds of MB per layer) are drawn with
torch's generator directly on the target device; host copies of sampled
layers are taken from those same tensors.
"""
from __future__ import annotations

from dataclasses import dataclass
from statistics import NormalDist

import numpy as np

F32 = 0
BF16 = 1
DTYPE_NAMES = {F32: "f32", BF16: "bf16"}


def gate_bias_for_gate_fraction(p_gate: float) -> float:
    """Gate bias b with P(N(b, 1) > 0) = p_gate (p_gate=1 maps to b=+8)."""
    if p_gate >= 1.0:
        return 8.0
    if p_gate <= 0.0:
        return -100.0
    return NormalDist().inv_cdf(p_gate)


def gate_bias_for_combined_sparsity(s: float) -> float:
    """Gate bias giving an expected fraction s of zero Combined activations.

    Combined_i is non-zero with probability Phi(b) * 1/2, so s = 1 - Phi(b)/2.
    s = 0.5 needs every gate open; that point uses b = +8.
    """
    return gate_bias_for_gate_fraction(2.0 * (1.0 - s))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounding = ((u >> 16) & 1) + 0x7FFF
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass
class FFNInputs:
    """One dReLU FFN layer's inputs (numpy, host)."""
    x: np.ndarray            # float32 [B][H]
    w_gate: np.ndarray       # float32 or uint16 (bf16 bits) [I][H]
    w_up: np.ndarray
    w_down_t: np.ndarray
    dtype: int               # F32 or BF16
    gate_bias: float | np.ndarray

    @property
    def shape(self):
        return self.x.shape[0], self.x.shape[1], self.w_gate.shape[0]


@dataclass
class MoEInputs:
    x: np.ndarray            # float32 [B][H]
    w_router: np.ndarray     # [E][H]
    w_gate: np.ndarray       # [E][I][H]
    w_up: np.ndarray
    w_down_t: np.ndarray
    dtype: int
    top_k: int
    gate_bias: float

    @property
    def shape(self):
        B, H = self.x.shape
        E, I, _ = self.w_gate.shape
        return B, H, I, E, self.top_k


def _store(a64: np.ndarray, dtype: int) -> np.ndarray:
    a32 = a64.astype(np.float32)
    return a32 if dtype == F32 else f32_to_bf16_bits(a32)


def _bias_column(b, I):
    b = np.asarray(b, dtype=np.float64)
    return np.broadcast_to(b, (I,)).astype(np.float64)


def make_ffn(batch: int, hidden: int, inter: int, gate_bias=-0.84, dtype: int = F32,
             seed=0, bias_feature: bool = True) -> FFNInputs:
    """Draw one FFN layer.  Draw order: x, W_gate, W_up, W_down_t."""
    rng = np.random.default_rng(seed)
    s = 1.0 / np.sqrt(hidden)
    x = rng.standard_normal((batch, hidden))
    wg = rng.standard_normal((inter, hidden)) * s
    wu = rng.standard_normal((inter, hidden)) * s
    wd = rng.standard_normal((inter, hidden)) * s
    if bias_feature:
        x[:, 0] = 1.0
        wg[:, 0] = _bias_column(gate_bias, inter)
    return FFNInputs(x=x.astype(np.float32), w_gate=_store(wg, dtype), w_up=_store(wu, dtype),
                     w_down_t=_store(wd, dtype), dtype=dtype, gate_bias=gate_bias)


def make_moe(batch: int, hidden: int, inter: int, n_experts: int, top_k: int,
             gate_bias=-1.5548, dtype: int = F32, seed=0) -> MoEInputs:
    """Draw one MoE layer.  Draw order: x, W_r, then per expert W_gate, W_up, W_down_t."""
    rng = np.random.default_rng(seed)
    s = 1.0 / np.sqrt(hidden)
    x = rng.standard_normal((batch, hidden))
    x[:, 0] = 1.0
    wr = rng.standard_normal((n_experts, hidden)) * s
    wg = np.empty((n_experts, inter, hidden))
    wu = np.empty_like(wg)
    wd = np.empty_like(wg)
    for e in range(n_experts):
        wg[e] = rng.standard_normal((inter, hidden)) * s
        wu[e] = rng.standard_normal((inter, hidden)) * s
        wd[e] = rng.standard_normal((inter, hidden)) * s
        wg[e][:, 0] = _bias_column(gate_bias, inter)
    return MoEInputs(x=x.astype(np.float32), w_router=_store(wr, dtype), w_gate=_store(wg, dtype),
                     w_up=_store(wu, dtype), w_down_t=_store(wd, dtype), dtype=dtype,
                     top_k=top_k, gate_bias=gate_bias)


def hot_cold_bias(inter: int, seed=0, hot_fraction=1.0 / 3.0, b_hot=0.2533, b_cold=-4.0) -> np.ndarray:
    """Per-neuron gate bias for a skewed workload: a random third of the
    neurons ("hot") open with probability Phi(0.2533) ~= 0.6, the rest almost
    never.  Per-token Combined sparsity stays ~90% while the union over a batch
    of independent tokens stays ~67% sparse."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 0x4C07]))
    hot = rng.random(inter) < hot_fraction
    return np.where(hot, b_hot, b_cold)


# ----------------------------------------------------------------------------
# Large stacks drawn on the device with torch (torch is only a memory / RNG
# provider here).


def torch_dtype(dtype: int):
    import torch
    return torch.float32 if dtype == F32 else torch.bfloat16


def make_ffn_stack_torch(n_layers: int, batch: int, hidden: int, inter: int, gate_bias=-0.8416,
                         dtype: int = BF16, seed=0, device="cuda"):
    """Draw n_layers independent FFN layers on `device`.

    Returns dict of tensors: x [L][B][H] f32, w_gate/w_up/w_down_t [L][I][H].
    Layer l is drawn from torch.Generator seeded with (seed * 1000003 + l).
    """
    import torch
    td = torch_dtype(dtype)
    s = 1.0 / float(np.sqrt(hidden))
    xs, wgs, wus, wds = [], [], [], []
    bias = torch.as_tensor(np.asarray(gate_bias, dtype=np.float32), device=device)
    for l in range(n_layers):
        g = torch.Generator(device=device)
        g.manual_seed(int(seed) * 1000003 + l)
        x = torch.randn(batch, hidden, generator=g, device=device, dtype=torch.float32)
        x[:, 0] = 1.0
        wg = torch.randn(inter, hidden, generator=g, device=device, dtype=torch.float32).mul_(s)
        wg[:, 0] = bias
        wu = torch.randn(inter, hidden, generator=g, device=device, dtype=torch.float32).mul_(s)
        wd = torch.randn(inter, hidden, generator=g, device=device, dtype=torch.float32).mul_(s)
        xs.append(x)
        wgs.append(wg.to(td))
        del wg
        wus.append(wu.to(td))
        del wu
        wds.append(wd.to(td))
        del wd
    return {"x": torch.stack(xs), "w_gate": wgs, "w_up": wus, "w_down_t": wds}


def make_moe_stack_torch(n_layers: int, batch: int, hidden: int, inter: int, n_experts: int,
                         top_k: int, gate_bias=-1.5548, dtype: int = BF16, seed=0, device="cuda"):
    """Draw n_layers independent MoE layers on `device` (packed [E][I][H] experts)."""
    import torch
    td = torch_dtype(dtype)
    s = 1.0 / float(np.sqrt(hidden))
    out = {"x": [], "w_router": [], "w_gate": [], "w_up": [], "w_down_t": []}
    for l in range(n_layers):
        g = torch.Generator(device=device)
        g.manual_seed(int(seed) * 1000003 + 7919 * (l + 1))
        x = torch.randn(batch, hidden, generator=g, device=device, dtype=torch.float32)
        x[:, 0] = 1.0
        wr = torch.randn(n_experts, hidden, generator=g, device=device).mul_(s)
        packs = []
        for name in ("w_gate", "w_up", "w_down_t"):
            t = torch.empty(n_experts, inter, hidden, device=device, dtype=td)
            for e in range(n_experts):
                w = torch.randn(inter, hidden, generator=g, device=device).mul_(s)
                if name == "w_gate":
                    w[:, 0] = float(gate_bias)
                t[e].copy_(w)
                del w
            packs.append(t)
        out["x"].append(x)
        out["w_router"].append(wr.to(td))
        for name, t in zip(("w_gate", "w_up", "w_down_t"), packs):
            out[name].append(t)
    out["x"] = torch.stack(out["x"])
    return out


def tensor_to_host_array(t, dtype: int) -> np.ndarray:
    """Host numpy copy of a device tensor in the oracle's storage format."""
    import torch
    t = t.detach().to("cpu").contiguous()
    if dtype == BF16:
        return t.view(torch.int16).numpy().view(np.uint16).copy()
    return t.numpy().astype(np.float32, copy=True)
