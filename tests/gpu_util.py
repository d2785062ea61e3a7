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
