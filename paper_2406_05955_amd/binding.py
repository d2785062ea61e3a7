"""Thin ctypes binding of libturbosparse.so (include/turbosparse.h).

Argument marshalling only: torch tensors supply device memory and the
stream; every step of the FFN runs in the library's HIP kernels.  There is no
fallback: if the library is missing this module raises on import.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libturbosparse.so")

TS_F32 = 0
TS_BF16 = 1

STATUS = {0: "TS_OK", 1: "TS_ERR_NULL", 2: "TS_ERR_SHAPE", 3: "TS_ERR_DTYPE", 4: "TS_ERR_ALIGN",
          5: "TS_ERR_WORKSPACE", 6: "TS_ERR_HIP", 7: "TS_ERR_UNSUPPORTED"}

EXPORTED = ["ts_ffn_workspace_bytes", "ts_ffn_sparse", "ts_ffn_sparse_act", "ts_ffn_sparse_topk", "ts_ffn_dense",
            "ts_ffn_given_workspace_bytes", "ts_ffn_sparse_noalloc",
            "ts_ffn_sparse_given", "ts_moe_workspace_bytes", "ts_moe_sparse",
            "ts_moe_dense", "ts_status_str", "ts_last_error", "ts_version", "ts_prof_enable", "ts_prof_reset",
            "ts_prof_read", "ts_probe_read", "ts_probe_copy", "ts_tune_set"]


class TSError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str = ""):
        self.code = code
        super().__init__(f"{where}: {STATUS.get(code, code)}" + (f" ({detail})" if detail else ""))


class ffn_stats_t(ctypes.Structure):
    _fields_ = [("n_gate", ctypes.c_void_p), ("n_active", ctypes.c_void_p), ("gate_idx", ctypes.c_void_p),
                ("active_idx", ctypes.c_void_p), ("n_union", ctypes.c_void_p)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2406_05955_amd.build` "
                          "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    st = ctypes.c_int
    lib.ts_ffn_workspace_bytes.argtypes = [i, i, i, i]
    lib.ts_ffn_workspace_bytes.restype = sz
    lib.ts_ffn_sparse.argtypes = [vp, vp, vp, vp, i, i, i, i, vp, vp, vp, sz, vp]
    lib.ts_ffn_sparse.restype = st
    lib.ts_ffn_sparse_noalloc.argtypes = [vp, vp, vp, vp, i, i, i, i, vp, vp, vp]
    lib.ts_ffn_sparse_noalloc.restype = st
    lib.ts_ffn_dense.argtypes = [vp, vp, vp, vp, i, i, i, i, vp, vp, sz, vp]
    lib.ts_ffn_dense.restype = st
    lib.ts_ffn_sparse_act.argtypes = [vp, vp, vp, vp, i, i, i, i, i, ctypes.c_float, vp, vp, vp, sz, vp]
    lib.ts_ffn_sparse_act.restype = st
    lib.ts_ffn_sparse_topk.argtypes = [vp, vp, vp, vp, i, i, i, i, i, vp, vp, vp, sz, vp]
    lib.ts_ffn_sparse_topk.restype = st
    lib.ts_ffn_given_workspace_bytes.argtypes = [i, i, i, i, i]
    lib.ts_ffn_given_workspace_bytes.restype = sz
    lib.ts_ffn_sparse_given.argtypes = [vp, vp, vp, vp, i, i, i, i, vp, vp, i, vp, vp, vp, sz, vp]
    lib.ts_ffn_sparse_given.restype = st
    lib.ts_moe_workspace_bytes.argtypes = [i, i, i, i, i, i]
    lib.ts_moe_workspace_bytes.restype = sz
    lib.ts_moe_sparse.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, vp, vp, vp, vp, sz, vp]
    lib.ts_moe_sparse.restype = st
    lib.ts_moe_dense.argtypes = [vp, vp, vp, vp, vp, i, i, i, i, i, i, vp, vp, vp, vp, sz, vp]
    lib.ts_moe_dense.restype = st
    lib.ts_status_str.argtypes = [st]
    lib.ts_status_str.restype = ctypes.c_char_p
    lib.ts_last_error.argtypes = []
    lib.ts_last_error.restype = ctypes.c_char_p
    lib.ts_version.argtypes = []
    lib.ts_version.restype = ctypes.c_char_p
    lib.ts_prof_enable.argtypes = [i]
    lib.ts_prof_enable.restype = None
    lib.ts_prof_reset.argtypes = []
    lib.ts_prof_reset.restype = None
    lib.ts_prof_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_long), ctypes.POINTER(ctypes.c_double)]
    lib.ts_prof_read.restype = st
    lib.ts_probe_read.argtypes = [vp, sz, vp, vp]
    lib.ts_probe_read.restype = st
    lib.ts_probe_copy.argtypes = [vp, vp, sz, vp]
    lib.ts_probe_copy.restype = st
    lib.ts_tune_set.argtypes = [ctypes.c_char_p, i]
    lib.ts_tune_set.restype = st
    return lib


lib = _load()


def _check(code: int, where: str):
    if code != 0:
        # the HIP message; the allocation-free entry point also explains a
        # shape beyond its scratch array there
        own = where == "ts_ffn_sparse_noalloc" and code in (5, 7)
        detail = lib.ts_last_error().decode() if code == 6 or own else ""
        raise TSError(code, where, detail)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def wdtype_of(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return TS_F32
    if t.dtype == torch.bfloat16:
        return TS_BF16
    raise TypeError(f"weights must be float32 or bfloat16, got {t.dtype}")


def _need_cuda(*ts):
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("tensors must be contiguous device tensors")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError(f"tensors on different devices ({dev}, {t.device})")


def _check_tensors(x, w_gate, w_up, w_down_t, out, w_router=None):
    """What the C ABI cannot check (it sees only pointers and the sizes passed
    with them): x float32 [B][H]; W_gate, W_up, W_down_t one dtype and one
    shape, [I][H] or, for the MoE layer, [E][I][H] with the router [E][H] of
    the same dtype; out float32 [B][H]; all contiguous on one device.  A
    mismatch here would let the kernels read or write past a buffer."""
    if x.dtype != torch.float32 or x.dim() != 2:
        raise TypeError(f"x must be a float32 [batch][hidden] tensor, got {x.dtype} {tuple(x.shape)}")
    B, H = x.shape
    moe = w_router is not None
    wdtype_of(w_gate)
    if w_gate.dim() != (3 if moe else 2) or w_gate.shape[-1] != H:
        raise ValueError(f"w_gate must be [{'experts][' if moe else ''}inter][{H}], got {tuple(w_gate.shape)}")
    for name, w in (("w_up", w_up), ("w_down_t", w_down_t)):
        if w.dtype != w_gate.dtype or w.shape != w_gate.shape:
            raise ValueError(f"{name} must match w_gate ({w_gate.dtype} {tuple(w_gate.shape)}), "
                             f"got {w.dtype} {tuple(w.shape)}")
    if moe and (w_router.dtype != w_gate.dtype or tuple(w_router.shape) != (w_gate.shape[0], H)):
        raise ValueError(f"w_router must be {w_gate.dtype} [{w_gate.shape[0]}][{H}], "
                         f"got {w_router.dtype} {tuple(w_router.shape)}")
    if out is not None and (out.dtype != torch.float32 or tuple(out.shape) != (B, H)):
        raise ValueError(f"out must be float32 [{B}][{H}], got {out.dtype} {tuple(out.shape)}")
    _need_cuda(x, out, w_gate, w_up, w_down_t, w_router)


def ffn_workspace_bytes(batch: int, hidden: int, inter: int, wdtype: int) -> int:
    return int(lib.ts_ffn_workspace_bytes(batch, hidden, inter, wdtype))


def ffn_given_workspace_bytes(batch: int, hidden: int, inter: int, max_count: int, wdtype: int) -> int:
    return int(lib.ts_ffn_given_workspace_bytes(batch, hidden, inter, max_count, wdtype))


def moe_workspace_bytes(batch: int, hidden: int, inter: int, n_experts: int, top_k: int, wdtype: int) -> int:
    return int(lib.ts_moe_workspace_bytes(batch, hidden, inter, n_experts, top_k, wdtype))


def _workspace(nbytes: int, device, ws):
    """The caller's workspace (any dtype; its size in bytes is passed on), or
    a new one of the size the library asks for."""
    if ws is not None:
        _need_cuda(ws)
        if ws.device != device:
            raise ValueError(f"workspace on {ws.device}, tensors on {device}")
        return ws
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


def _nbytes(t):
    return t.numel() * t.element_size()


def _stats_struct(batch_slots: int, inter: int, device, want: bool):
    if not want:
        return None, None
    d = {
        "n_gate": torch.empty(batch_slots, dtype=torch.int32, device=device),
        "n_active": torch.empty(batch_slots, dtype=torch.int32, device=device),
        "gate_idx": torch.empty(batch_slots, inter, dtype=torch.int32, device=device),
        "active_idx": torch.empty(batch_slots, inter, dtype=torch.int32, device=device),
    }
    s = ffn_stats_t(_ptr(d["n_gate"]), _ptr(d["n_active"]), _ptr(d["gate_idx"]), _ptr(d["active_idx"]), None)
    return s, d


def ffn_sparse(x, w_gate, w_up, w_down_t, out=None, stats: bool = False, union: bool = False, ws=None,
               stream=None):
    """ts_ffn_sparse.  x [B][H] f32; weights [I][H] f32/bf16.  Returns out, or
    (out, stats dict) when stats/union is requested."""
    _check_tensors(x, w_gate, w_up, w_down_t, out)
    B, H = x.shape
    I = w_gate.shape[0]
    dt = wdtype_of(w_gate)
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    ws = _workspace(ffn_workspace_bytes(B, H, I, dt), x.device, ws)
    st, d = _stats_struct(B, I, x.device, stats or union)
    if union:
        d["n_union"] = torch.empty(2, dtype=torch.int32, device=x.device)
        st.n_union = _ptr(d["n_union"])
    code = lib.ts_ffn_sparse(_ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, _ptr(out),
                             ctypes.byref(st) if st is not None else None, _ptr(ws), _nbytes(ws), _stream(stream))
    _check(code, "ts_ffn_sparse")
    return (out, d) if d is not None else out


# the fixed scratch array of ts_ffn_sparse_noalloc (TS_NOALLOC_SCRATCH_BYTES)
NOALLOC_SCRATCH_BYTES = 32 << 20


def ffn_sparse_noalloc(x, w_gate, w_up, w_down_t, out=None, stats: bool = False, union: bool = False,
                       stream=None):
    """ts_ffn_sparse_noalloc: ts_ffn_sparse with the library's fixed scratch
    array instead of a workspace.  Pass `out` to make the call allocate
    nothing on the Python side either.  Returns out, or (out, stats dict)."""
    _check_tensors(x, w_gate, w_up, w_down_t, out)
    B, H = x.shape
    I = w_gate.shape[0]
    dt = wdtype_of(w_gate)
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    st, d = _stats_struct(B, I, x.device, stats or union)
    if union:
        d["n_union"] = torch.empty(2, dtype=torch.int32, device=x.device)
        st.n_union = _ptr(d["n_union"])
    code = lib.ts_ffn_sparse_noalloc(_ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, _ptr(out),
                                     ctypes.byref(st) if st is not None else None, _stream(stream))
    _check(code, "ts_ffn_sparse_noalloc")
    return (out, d) if d is not None else out


TS_ACT_DRELU = 0
TS_ACT_RELU_GATE = 1


def ffn_sparse_act(x, w_gate, w_up, w_down_t, act: int, tau: float = 0.0, out=None, stats: bool = False,
                   union: bool = False, ws=None, stream=None):
    """ts_ffn_sparse_act: act TS_ACT_DRELU (tau 0) or TS_ACT_RELU_GATE
    (Combined = max(0, gate - tau) * up).  Returns out, or (out, stats dict)."""
    _check_tensors(x, w_gate, w_up, w_down_t, out)
    B, H = x.shape
    I = w_gate.shape[0]
    dt = wdtype_of(w_gate)
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    ws = _workspace(ffn_workspace_bytes(B, H, I, dt), x.device, ws)
    st, d = _stats_struct(B, I, x.device, stats or union)
    if union:
        d["n_union"] = torch.empty(2, dtype=torch.int32, device=x.device)
        st.n_union = _ptr(d["n_union"])
    code = lib.ts_ffn_sparse_act(_ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, int(act),
                                 float(tau), _ptr(out), ctypes.byref(st) if st is not None else None, _ptr(ws),
                                 _nbytes(ws), _stream(stream))
    _check(code, "ts_ffn_sparse_act")
    return (out, d) if d is not None else out


def ffn_sparse_topk(x, w_gate, w_up, w_down_t, keep: int, out=None, stats: bool = False, ws=None, stream=None):
    """ts_ffn_sparse_topk: dReLU FFN keeping each token's `keep` largest
    Combined activations.  Returns out, or (out, stats dict)."""
    _check_tensors(x, w_gate, w_up, w_down_t, out)
    B, H = x.shape
    I = w_gate.shape[0]
    dt = wdtype_of(w_gate)
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    ws = _workspace(ffn_workspace_bytes(B, H, I, dt), x.device, ws)
    st, d = _stats_struct(B, I, x.device, stats)
    code = lib.ts_ffn_sparse_topk(_ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, int(keep),
                                  _ptr(out), ctypes.byref(st) if st is not None else None, _ptr(ws), _nbytes(ws),
                                  _stream(stream))
    _check(code, "ts_ffn_sparse_topk")
    return (out, d) if d is not None else out


def ffn_dense(x, w_gate, w_up, w_down_t, out=None, ws=None, stream=None):
    """ts_ffn_dense (all neurons, all three matrices read)."""
    _check_tensors(x, w_gate, w_up, w_down_t, out)
    B, H = x.shape
    I = w_gate.shape[0]
    dt = wdtype_of(w_gate)
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    ws = _workspace(ffn_workspace_bytes(B, H, I, dt), x.device, ws)
    code = lib.ts_ffn_dense(_ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, _ptr(out), _ptr(ws),
                            _nbytes(ws), _stream(stream))
    _check(code, "ts_ffn_dense")
    return out


def ffn_sparse_given(x, w_gate, w_up, w_down_t, idx, count, out=None, stats: bool = False, ws=None, stream=None):
    """ts_ffn_sparse_given: the FFN over given neuron lists.  idx int32
    [B][max_count], count int32 [B] (device tensors).  Returns out, or (out,
    {"n_gate", "n_active"}) with stats=True."""
    _check_tensors(x, w_gate, w_up, w_down_t, out)
    _need_cuda(x, idx, count)
    B, H = x.shape
    I = w_gate.shape[0]
    dt = wdtype_of(w_gate)
    if idx.dim() != 2 or idx.shape[0] != B or count.numel() != B:
        raise ValueError("idx must be [batch][max_count] and count [batch]")
    if idx.dtype != torch.int32 or count.dtype != torch.int32:
        raise TypeError("idx and count must be int32")
    maxc = idx.shape[1]
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    ws = _workspace(ffn_given_workspace_bytes(B, H, I, maxc, dt), x.device, ws)
    d = st = None
    if stats:
        d = {"n_gate": torch.empty(B, dtype=torch.int32, device=x.device),
             "n_active": torch.empty(B, dtype=torch.int32, device=x.device)}
        st = ffn_stats_t(_ptr(d["n_gate"]), _ptr(d["n_active"]), None, None, None)
    code = lib.ts_ffn_sparse_given(_ptr(x), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, _ptr(idx),
                                   _ptr(count), maxc, _ptr(out), ctypes.byref(st) if st is not None else None,
                                   _ptr(ws), _nbytes(ws), _stream(stream))
    _check(code, "ts_ffn_sparse_given")
    return (out, d) if d is not None else out


def moe_sparse(x, w_router, w_gate, w_up, w_down_t, top_k: int, out=None, stats: bool = False, ws=None,
               stream=None, dense: bool = False):
    """ts_moe_sparse (or ts_moe_dense with dense=True).  Returns
    (out, topk_idx, topk_w) or (out, topk_idx, topk_w, stats dict)."""
    _check_tensors(x, w_gate, w_up, w_down_t, out, w_router=w_router)
    B, H = x.shape
    E, I = w_gate.shape[0], w_gate.shape[1]
    dt = wdtype_of(w_gate)
    if out is None:
        out = torch.empty(B, H, dtype=torch.float32, device=x.device)
    idx = torch.empty(B, top_k, dtype=torch.int32, device=x.device)
    wts = torch.empty(B, top_k, dtype=torch.float32, device=x.device)
    ws = _workspace(moe_workspace_bytes(B, H, I, E, top_k, dt), x.device, ws)
    if dense:
        code = lib.ts_moe_dense(_ptr(x), _ptr(w_router), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, E,
                                top_k, _ptr(out), _ptr(idx), _ptr(wts), _ptr(ws), _nbytes(ws), _stream(stream))
        _check(code, "ts_moe_dense")
        return out, idx, wts
    st, d = _stats_struct(B * top_k, I, x.device, stats)
    code = lib.ts_moe_sparse(_ptr(x), _ptr(w_router), _ptr(w_gate), _ptr(w_up), _ptr(w_down_t), dt, B, H, I, E,
                             top_k, _ptr(out), _ptr(idx), _ptr(wts), ctypes.byref(st) if st is not None else None,
                             _ptr(ws), _nbytes(ws), _stream(stream))
    _check(code, "ts_moe_sparse")
    return (out, idx, wts, d) if d is not None else (out, idx, wts)


def moe_dense(x, w_router, w_gate, w_up, w_down_t, top_k: int, out=None, ws=None, stream=None):
    return moe_sparse(x, w_router, w_gate, w_up, w_down_t, top_k, out=out, ws=ws, stream=stream, dense=True)


def probe_read(src: torch.Tensor, sink: torch.Tensor, stream=None):
    """ts_probe_read: sink holds one float32 per workgroup (4096)."""
    if sink.dtype != torch.float32 or sink.numel() < 4096:
        raise ValueError("sink must be float32 with at least 4096 elements")
    _need_cuda(src, sink)
    _check(lib.ts_probe_read(_ptr(src), _nbytes(src), _ptr(sink), _stream(stream)), "ts_probe_read")


def probe_copy(src: torch.Tensor, dst: torch.Tensor, stream=None):
    """ts_probe_copy: copies all of src into the start of dst."""
    if _nbytes(dst) < _nbytes(src):
        raise ValueError("dst is smaller than src")
    _need_cuda(src, dst)
    _check(lib.ts_probe_copy(_ptr(src), _ptr(dst), _nbytes(src), _stream(stream)), "ts_probe_copy")


def prof_enable(on: bool):
    lib.ts_prof_enable(1 if on else 0)


def prof_reset():
    lib.ts_prof_reset()


def prof_read(kernel: str):
    n = ctypes.c_long()
    ms = ctypes.c_double()
    _check(lib.ts_prof_read(kernel.encode(), ctypes.byref(n), ctypes.byref(ms)), "ts_prof_read")
    return int(n.value), float(ms.value)


def tune_set(key: str, value: int):
    _check(lib.ts_tune_set(key.encode(), int(value)), "ts_tune_set")


def version() -> str:
    return lib.ts_version().decode()
