"""Plant plausible mistakes in copies of oracle.c (on the CPU) and check that
at least one pin rejects every mutant, so the pins are strong enough to catch
a dropped term, a wrong sign or index, a transposed operand, a missing ReLU,
a wrong tie-break or a missing renormalisation."""
import os
import subprocess

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")

MUTANTS = {
    "gate_only_relu": ("h[i] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;", "h[i] = (sg > 0.0) ? sg * su : 0.0;"),
    "no_relu": ("h[i] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;", "h[i] = sg * su;"),
    "up_only_relu": ("h[i] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;", "h[i] = (su > 0.0) ? sg * su : 0.0;"),
    "dropped_bias_column": ("for (int j = 0; j < H; ++j) {\n            double xj",
                            "for (int j = 1; j < H; ++j) {\n            double xj"),
    "up_reads_gate": ("su += load_w(wu, dtype, row + j) * xj;", "su += load_w(wg, dtype, row + j) * xj;"),
    "down_transposed": ("y[j] += load_w(wdt, dtype, row + j) * hv;",
                        "y[j] += load_w(wdt, dtype, (size_t)j * (size_t)I + ii) * hv;"),
    "bf16_shift": ("<< 16;", "<< 15;"),
    "softmax_sign": ("probs[e] = exp(logits[e] - m);", "probs[e] = exp(m - logits[e]);"),
    "tie_upper_index": ("probs[e] > probs[best]", "probs[e] >= probs[best]"),
    "no_renormalise": ("w[k] = probs[idx[k]] / psum;", "w[k] = probs[idx[k]];"),
    "moe_wrong_expert_down": ("const char *base_d = (const char *)wdt + (size_t)e * expert_bytes;",
                              "const char *base_d = (const char *)wdt;"),
    "moe_rank_weight_swap": ("yt[j] += w[rank] * ye[j];", "yt[j] += w[K - 1 - rank] * ye[j];"),
    "act_shift_sign": ("ha[i] = sg > tau ? (sg - tau) * su : 0.0;", "ha[i] = sg > tau ? (sg + tau) * su : 0.0;"),
    "act_unshifted_product": ("ha[i] = sg > tau ? (sg - tau) * su : 0.0;", "ha[i] = sg > tau ? sg * su : 0.0;"),
    "act_up_masked": ("ha[i] = sg > tau ? (sg - tau) * su : 0.0;",
                      "ha[i] = (sg > tau && su > 0.0) ? (sg - tau) * su : 0.0;"),
    "topk_tie_upper_index": ("return (a > b) - (a < b);", "return (a < b) - (a > b);"),
    "topk_smallest_first": ("    if (va > vb)\n        return -1;\n    if (va < vb)\n        return 1;",
                            "    if (va > vb)\n        return 1;\n    if (va < vb)\n        return -1;"),
    "topk_off_by_one": ("int k = keep < I ? keep : I, nk = 0;", "int k = keep < I ? keep + 1 : I, nk = 0;"),
    "given_gate_only_relu": ("hl[k] = (sg > 0.0 && su > 0.0) ? sg * su : 0.0;", "hl[k] = (sg > 0.0) ? sg * su : 0.0;"),
    "given_count_ignored": ("int n = count[t] < 0 ? 0 : (count[t] > maxc ? maxc : count[t]);", "int n = maxc;"),
    "given_down_list_position": ("double hv = hl[kk];\n                size_t row = (size_t)i * (size_t)H;",
                                 "double hv = hl[kk];\n                size_t row = (size_t)kk * (size_t)H;"),
    "given_repeat_dropped": ("for (int kk = 0; kk < n; ++kk) {\n                int i = lt[kk];\n                if (i < 0 || i >= I)\n                    continue;",
                             "for (int kk = 0; kk < n; ++kk) {\n                int i = lt[kk];\n                if (i < 0 || i >= I || (kk > 0 && lt[kk - 1] == i) || (kk > 1 && lt[kk - 2] == i))\n                    continue;"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    mutated = src.replace(old, new)
    c = tmp_path / "oracle_mut.c"
    c.write_text(mutated)
    so = tmp_path / "liboracle_mut.so"
    subprocess.run(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-o", str(so),
                    str(c), "-lm"], check=True)
    lib = oracle.load_library(str(so))
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(lib)
        except AssertionError:
            caught.append(pin.__name__)
    assert caught, f"no pin rejects mutant {name}"
