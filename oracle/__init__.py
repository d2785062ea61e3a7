"""fp64 CPU oracle for the dReLU FFN and its MoE form (Turbo Sparse,
arXiv 2406.05955, Eq. gated-MLP, Eq. drelu, section 6.2).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the HIP library: the arithmetic is in ``oracle.c`` (plain C, fp64, fixed
summation order), loaded here through ctypes.

Parity status: every function here is pinned by CPU tests against values that
do not come from the oracle itself (a hand-worked example, exact rational
arithmetic on tiny inputs within the fp64 forward-error bound, library special
cases and exact invariants).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

F32 = 0
BF16 = 1


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (OpenMP, no FMA contraction)."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


def _bind(lib):
    vp, ip, dp = ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p
    lib.or_ffn.argtypes = [vp, vp, vp, vp, ip, ip, ip, ip, dp, dp, dp, ip]
    lib.or_ffn.restype = ctypes.c_int
    lib.or_moe.argtypes = [vp, vp, vp, vp, vp, ip, ip, ip, ip, ip, ip, dp, vp, dp, dp, dp, dp, ip]
    lib.or_moe.restype = ctypes.c_int
    lib.or_ffn_given.argtypes = [vp, vp, vp, vp, ip, ip, ip, ip, vp, vp, ip, dp, vp, vp, ip]
    lib.or_ffn_given.restype = ctypes.c_int
    lib.or_ffn_act.argtypes = [vp, vp, vp, vp, ip, ip, ip, ip, ip, ctypes.c_double, dp, dp, dp, ip]
    lib.or_ffn_act.restype = ctypes.c_int
    lib.or_ffn_topk.argtypes = [vp, vp, vp, vp, ip, ip, ip, ip, ip, dp, vp, ip]
    lib.or_ffn_topk.restype = ctypes.c_int
    lib.or_max_threads.argtypes = []
    lib.or_max_threads.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    if _lib is None:
        build()
        _lib = _bind(ctypes.CDLL(_LIB))
    return _lib


def load_library(path: str):
    """Bind another build of oracle.c (the mutation tests compile planted-bug
    variants and check that the pins reject them)."""
    return _bind(ctypes.CDLL(os.path.abspath(path)))


def max_threads() -> int:
    return _load().or_max_threads()


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _weights(a, dtype):
    want = np.float32 if dtype == F32 else np.uint16
    a = np.ascontiguousarray(a)
    if a.dtype != want:
        raise TypeError(f"weights must be {want} for dtype {dtype}, got {a.dtype}")
    return a


@dataclass
class FFNResult:
    y: np.ndarray       # fp64 [B][H]
    g: np.ndarray       # fp64 [B][I] gate projection before ReLU
    u: np.ndarray       # fp64 [B][I] up projection before ReLU

    def gate_set(self, t: int) -> np.ndarray:
        """G_t: neurons whose gate projection is strictly positive (ascending)."""
        return np.nonzero(self.g[t] > 0.0)[0].astype(np.int32)

    def active_set(self, t: int) -> np.ndarray:
        """A_t: neurons whose dReLU Combined activation is non-zero (ascending)."""
        return np.nonzero((self.g[t] > 0.0) & (self.u[t] > 0.0))[0].astype(np.int32)

    @property
    def n_gate(self) -> np.ndarray:
        return (self.g > 0.0).sum(axis=1).astype(np.int32)

    @property
    def n_active(self) -> np.ndarray:
        return ((self.g > 0.0) & (self.u > 0.0)).sum(axis=1).astype(np.int32)


def ffn(x, w_gate, w_up, w_down_t, dtype: int, threads: int = 0, lib=None) -> FFNResult:
    """Dense dReLU FFN in fp64: y = W_down_t^T (max(0, W_gate x) * max(0, W_up x))."""
    lib = lib or _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    B, H = x.shape
    wg, wu, wd = (_weights(w, dtype) for w in (w_gate, w_up, w_down_t))
    I = wg.shape[0]
    for w in (wg, wu, wd):
        if w.shape != (I, H):
            raise ValueError(f"weight shape {w.shape} != {(I, H)}")
    y = np.empty((B, H), np.float64)
    g = np.empty((B, I), np.float64)
    u = np.empty((B, I), np.float64)
    rc = lib.or_ffn(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), dtype, B, H, I, _ptr(y), _ptr(g), _ptr(u),
                    int(threads))
    if rc != 0:
        raise RuntimeError("or_ffn failed")
    return FFNResult(y=y, g=g, u=u)


ACT_DRELU = 0
ACT_RELU_GATE = 1


@dataclass
class ActResult:
    y: np.ndarray       # fp64 [B][H]
    g: np.ndarray       # fp64 [B][I] gate projection before the activation
    u: np.ndarray       # fp64 [B][I] up projection
    act: int
    tau: float

    def gate_set(self, t: int) -> np.ndarray:
        """Neurons whose gate passes the activation's threshold (ascending)."""
        return np.nonzero(self.g[t] > self.tau)[0].astype(np.int32)

    def active_set(self, t: int) -> np.ndarray:
        """Neurons with a non-zero Combined activation (ascending)."""
        if self.act == ACT_DRELU:
            m = (self.g[t] > 0.0) & (self.u[t] > 0.0)
        else:
            m = (self.g[t] > self.tau) & (self.u[t] != 0.0)
        return np.nonzero(m)[0].astype(np.int32)


def ffn_act(x, w_gate, w_up, w_down_t, dtype: int, act: int, tau: float = 0.0, threads: int = 0,
            lib=None) -> ActResult:
    """FFN in fp64 with act 0 = dReLU (tau 0) or act 1 = gate-only ReLU with
    threshold tau: Combined = max(0, g - tau) * u (ReGLU at tau = 0)."""
    lib = lib or _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    B, H = x.shape
    wg, wu, wd = (_weights(w, dtype) for w in (w_gate, w_up, w_down_t))
    I = wg.shape[0]
    y = np.empty((B, H), np.float64)
    g = np.empty((B, I), np.float64)
    u = np.empty((B, I), np.float64)
    rc = lib.or_ffn_act(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), dtype, B, H, I, int(act), float(tau), _ptr(y),
                        _ptr(g), _ptr(u), int(threads))
    if rc != 0:
        raise RuntimeError("or_ffn_act failed")
    return ActResult(y=y, g=g, u=u, act=int(act), tau=float(tau))


def ffn_topk(x, w_gate, w_up, w_down_t, dtype: int, keep: int, threads: int = 0, lib=None):
    """dReLU FFN with the top-k magnitude mask in fp64: per token only the
    `keep` largest |Combined| (ties: lower index) contribute.  Returns (y
    [B][H], n_kept [B]: kept neurons with a non-zero activation)."""
    lib = lib or _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    B, H = x.shape
    wg, wu, wd = (_weights(w, dtype) for w in (w_gate, w_up, w_down_t))
    I = wg.shape[0]
    y = np.empty((B, H), np.float64)
    nk = np.empty(B, np.int32)
    rc = lib.or_ffn_topk(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), dtype, B, H, I, int(keep), _ptr(y), _ptr(nk),
                         int(threads))
    if rc != 0:
        raise RuntimeError("or_ffn_topk failed")
    return y, nk


@dataclass
class GivenResult:
    y: np.ndarray          # fp64 [B][H]
    n_open: np.ndarray     # int32 [B] listed entries with gate > 0
    n_active: np.ndarray   # int32 [B] listed entries with gate > 0 and up > 0


def ffn_given(x, w_gate, w_up, w_down_t, dtype: int, idx, count, threads: int = 0, lib=None) -> GivenResult:
    """dReLU FFN over given neuron lists in fp64 (list order; entries outside
    [0, I) skipped): y_t = sum over listed i of max(0, g_i) max(0, u_i) W_down_t[i]."""
    lib = lib or _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    B, H = x.shape
    wg, wu, wd = (_weights(w, dtype) for w in (w_gate, w_up, w_down_t))
    I = wg.shape[0]
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    if idx.ndim == 1:
        idx = idx[None, :]
    count = np.ascontiguousarray(count, dtype=np.int32).reshape(-1)
    if idx.shape[0] != B or count.shape[0] != B:
        raise ValueError("idx / count must have one row / entry per token")
    maxc = idx.shape[1]
    y = np.empty((B, H), np.float64)
    no = np.empty(B, np.int32)
    na = np.empty(B, np.int32)
    rc = lib.or_ffn_given(_ptr(x), _ptr(wg), _ptr(wu), _ptr(wd), dtype, B, H, I, _ptr(idx), _ptr(count), maxc,
                          _ptr(y), _ptr(no), _ptr(na), int(threads))
    if rc != 0:
        raise RuntimeError("or_ffn_given failed")
    return GivenResult(y=y, n_open=no, n_active=na)


@dataclass
class MoEResult:
    y: np.ndarray          # fp64 [B][H]
    topk_idx: np.ndarray   # int32 [B][K], rank order (largest probability first)
    topk_w: np.ndarray     # fp64 [B][K]
    probs: np.ndarray      # fp64 [B][E]
    g: np.ndarray          # fp64 [B][K][I] (rank order)
    u: np.ndarray          # fp64 [B][K][I]


def moe(x, w_router, w_gate, w_up, w_down_t, dtype: int, top_k: int, threads: int = 0,
        keep_projections: bool = True, lib=None) -> MoEResult:
    """MoE layer in fp64: softmax router, top-k, renormalised mixture of dReLU experts."""
    lib = lib or _load()
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim == 1:
        x = x[None, :]
    B, H = x.shape
    wr = _weights(w_router, dtype)
    wg, wu, wd = (_weights(w, dtype) for w in (w_gate, w_up, w_down_t))
    E, I = wg.shape[0], wg.shape[1]
    if wr.shape != (E, H):
        raise ValueError(f"router shape {wr.shape} != {(E, H)}")
    for w in (wg, wu, wd):
        if w.shape != (E, I, H):
            raise ValueError(f"expert weight shape {w.shape} != {(E, I, H)}")
    K = int(top_k)
    y = np.empty((B, H), np.float64)
    idx = np.empty((B, K), np.int32)
    wts = np.empty((B, K), np.float64)
    probs = np.empty((B, E), np.float64)
    g = np.empty((B, K, I), np.float64) if keep_projections else None
    u = np.empty((B, K, I), np.float64) if keep_projections else None
    rc = lib.or_moe(_ptr(x), _ptr(wr), _ptr(wg), _ptr(wu), _ptr(wd), dtype, B, H, I, E, K, _ptr(y),
                    _ptr(idx), _ptr(wts), _ptr(probs), _ptr(g), _ptr(u), int(threads))
    if rc != 0:
        raise RuntimeError("or_moe failed")
    return MoEResult(y=y, topk_idx=idx, topk_w=wts, probs=probs, g=g, u=u)
