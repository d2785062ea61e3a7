"""The C-ABI library on the CPU: it loads, exports every function that
include/turbosparse.h declares, and its host-side argument checks return the
documented status codes before anything is enqueued (no GPU is touched:
every call below is rejected during validation)."""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2406_05955_amd import binding as ts

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "turbosparse.h")

OK, NULL, SHAPE, DTYPE, ALIGN, WS, HIP, UNSUP = range(8)
A = 0x10000  # a 16-byte aligned fake device address; never dereferenced


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(ts_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_function():
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(ts.lib, n), n
    dyn = subprocess.run(["nm", "-D", "--defined-only", ts.LIB_PATH], capture_output=True, text=True).stdout
    for n in names:
        assert re.search(rf"\bT {n}$", dyn, flags=re.M), f"{n} not exported"
    assert set(ts.EXPORTED) == set(names)


def test_status_strings():
    for code in range(8):
        assert ts.lib.ts_status_str(code).decode().startswith(ts.STATUS[code])
    assert ts.version().startswith("turbosparse")


def _ffn(x=A, wg=A, wu=A, wd=A, dt=1, B=1, H=4096, I=14336, out=A, stats=None, ws=A, wsb=1 << 40):
    return ts.lib.ts_ffn_sparse(x, wg, wu, wd, dt, B, H, I, out, stats, ws, wsb, None)


def test_ffn_shape_checks():
    assert _ffn(B=0) == SHAPE
    assert _ffn(B=257) == SHAPE
    assert _ffn(I=0) == SHAPE
    assert _ffn(H=4100) == SHAPE            # bf16 needs hidden % 8 == 0
    assert _ffn(H=8200, dt=1) == SHAPE      # above 8192
    assert _ffn(H=4100, dt=0) == SHAPE      # fp32 above 4096
    assert _ffn(H=6, dt=0) == SHAPE
    assert _ffn(H=1026, dt=0) == SHAPE      # fp32 needs hidden % 4 == 0
    assert _ffn(dt=7) == DTYPE


def test_ffn_pointer_checks():
    assert _ffn(x=None) == NULL
    assert _ffn(wg=None) == NULL
    assert _ffn(wu=None) == NULL
    assert _ffn(wd=None) == NULL
    assert _ffn(out=None) == NULL
    assert _ffn(x=A + 4) == ALIGN
    assert _ffn(wd=A + 8) == ALIGN
    assert _ffn(out=A + 2) == ALIGN
    st = ts.ffn_stats_t(A + 2, None, None, None, None)
    assert _ffn(stats=ctypes.byref(st)) == ALIGN


def test_ffn_workspace_checks():
    need = ts.ffn_workspace_bytes(1, 4096, 14336, 1)
    assert need > 0
    assert _ffn(ws=None) == WS
    assert _ffn(wsb=need - 1) == WS
    assert _ffn(ws=A + 8, wsb=need) == ALIGN
    assert ts.ffn_workspace_bytes(0, 4096, 14336, 1) == 0
    assert ts.ffn_workspace_bytes(1, 4100, 14336, 1) == 0
    assert ts.lib.ts_ffn_dense(A, A, A, A, 1, 1, 4096, 14336, A, A, need - 1, None) == WS


def test_moe_checks():
    f = ts.lib.ts_moe_sparse

    def call(E=8, K=2, B=1, H=4096, I=14336, ws=A, wsb=1 << 40, idx=None, w=None, stats=None):
        return f(A, A, A, A, A, 1, B, H, I, E, K, A, idx, w, stats, ws, wsb, None)
    assert call(E=0) == SHAPE
    assert call(E=65) == SHAPE
    assert call(K=0) == SHAPE
    assert call(K=9, E=16) == SHAPE
    assert call(K=3, E=2) == SHAPE
    assert call(idx=A + 2) == ALIGN
    need = ts.moe_workspace_bytes(1, 4096, 14336, 8, 2, 1)
    assert need > 0
    assert call(wsb=need - 1) == WS
    st = ts.ffn_stats_t(None, None, None, None, A)
    assert call(stats=ctypes.byref(st)) == UNSUP
    assert f(A, None, A, A, A, 1, 1, 4096, 14336, 8, 2, A, None, None, None, A, need, None) == NULL


def test_probe_checks():
    assert ts.lib.ts_probe_read(None, 16, A, None) == NULL
    assert ts.lib.ts_probe_read(A, 15, A, None) == SHAPE
    assert ts.lib.ts_probe_copy(A, A + 4, 16, None) == ALIGN


def test_tune_checks():
    assert ts.lib.ts_tune_set(b"ffn_tile", 10) == SHAPE
    assert ts.lib.ts_tune_set(b"ffn_tile", 132) == SHAPE
    assert ts.lib.ts_tune_set(b"nope", 8) == SHAPE
    assert ts.lib.ts_tune_set(b"ffn_tile", 32) == OK
    assert ts.lib.ts_tune_set(b"ffn_interleave", 2) == SHAPE
    assert ts.lib.ts_tune_set(b"ffn_interleave", 1) == OK
    assert ts.lib.ts_tune_set(b"ffn_interleave", 0) == OK
    small = ts.ffn_workspace_bytes(1, 4096, 14336, 1)
    assert ts.lib.ts_tune_set(b"ffn_tile", 0) == OK
    assert ts.ffn_workspace_bytes(1, 4096, 14336, 1) < small


def test_given_checks():
    f = ts.lib.ts_ffn_sparse_given

    def call(x=A, dt=1, B=1, H=4096, I=14336, idx=A, cnt=A, maxc=3000, out=A, stats=None, ws=A, wsb=1 << 40):
        return f(x, A, A, A, dt, B, H, I, idx, cnt, maxc, out, stats, ws, wsb, None)
    need = ts.ffn_given_workspace_bytes(1, 4096, 14336, 3000, 1)
    assert need > 0
    assert ts.ffn_given_workspace_bytes(1, 4096, 14336, 0, 1) == 0
    # about one workgroup per compute unit: a 4-entry list needs one partial row
    assert ts.ffn_given_workspace_bytes(1, 4096, 14336, 4, 1) < need
    assert call(maxc=0) == SHAPE
    assert call(maxc=(1 << 24) + 1) == SHAPE
    assert call(B=0) == SHAPE
    assert call(dt=5) == DTYPE
    assert call(idx=None) == NULL
    assert call(cnt=None) == NULL
    assert call(x=None) == NULL
    assert call(idx=A + 2) == ALIGN
    assert call(cnt=A + 1) == ALIGN
    assert call(out=A + 4) == ALIGN
    assert call(wsb=need - 1) == WS
    assert call(ws=None) == WS
    # rows wider than the pipelined kernel serves (bf16 hidden 8192, fp32 hidden 4096)
    assert call(H=8192) == UNSUP
    assert call(H=4096, dt=0) == UNSUP
    # only the counts of the activity report are served
    st = ts.ffn_stats_t(None, None, A, None, None)
    assert call(stats=ctypes.byref(st)) == UNSUP
    st = ts.ffn_stats_t(None, None, None, None, A)
    assert call(stats=ctypes.byref(st)) == UNSUP
    st = ts.ffn_stats_t(A + 2, None, None, None, None)
    assert call(stats=ctypes.byref(st)) == ALIGN


def test_act_checks():
    f = ts.lib.ts_ffn_sparse_act

    def call(act=1, tau=0.0, B=1, H=4096, I=14336, out=A, ws=A, wsb=1 << 40, x=A):
        return f(x, A, A, A, 1, B, H, I, act, tau, out, None, ws, wsb, None)
    assert call(act=2) == SHAPE
    assert call(act=-1) == SHAPE
    assert call(act=0, tau=0.5) == SHAPE
    assert call(tau=float("nan")) == SHAPE
    assert call(tau=float("inf")) == SHAPE
    assert call(x=None) == NULL
    assert call(out=A + 4) == ALIGN
    need = ts.ffn_workspace_bytes(1, 4096, 14336, 1)
    assert call(wsb=need - 1) == WS
    assert call(act=0, wsb=need - 1) == WS
    assert call(B=0) == SHAPE


def test_topk_checks():
    f = ts.lib.ts_ffn_sparse_topk

    def call(keep=100, B=1, H=4096, I=14336, out=A, ws=A, wsb=1 << 40, stats=None):
        return f(A, A, A, A, 1, B, H, I, keep, out, stats, ws, wsb, None)
    assert call(keep=-1) == SHAPE
    assert call(I=16385) == UNSUP
    assert call(out=A + 8) == ALIGN
    need = ts.ffn_workspace_bytes(1, 4096, 14336, 1)
    assert call(wsb=need - 1) == WS
    assert call(B=0) == SHAPE


def test_c_program_links_the_library_only():
    """The plain-C ABI check links libturbosparse.so and the HIP runtime, and
    nothing of Python or PyTorch."""
    binp = os.path.join(ROOT, "tests", "c_abi", "_build", "c_smoke")
    if not os.path.exists(binp):
        pytest.skip("not built (__graft_entry__.build() builds it)")
    deps = subprocess.run(["ldd", binp], capture_output=True, text=True).stdout
    assert "libturbosparse.so" in deps and "not found" not in deps.split("libturbosparse.so")[1].split("\n")[0]
    assert "amdhip64" in deps
    assert "torch" not in deps and "python" not in deps


def test_noalloc_host_checks():
    """ts_ffn_sparse_noalloc runs ts_ffn_sparse's checks, then rejects a
    shape whose workspace exceeds its fixed scratch array, all before any
    HIP call (so these return on a machine without a GPU too)."""
    f = ts.lib.ts_ffn_sparse_noalloc
    assert f(A, A, A, A, 1, 8, 4096, 14336, A, None, None) == WS       # ~33 MiB > 32 MiB
    assert f(A, A, A, A, 1, 256, 4096, 14336, A, None, None) == WS
    assert f(A, A, A, A, 1, 0, 4096, 14336, A, None, None) == SHAPE
    assert f(None, A, A, A, 1, 1, 4096, 14336, A, None, None) == NULL
    assert f(A + 4, A, A, A, 1, 1, 4096, 14336, A, None, None) == ALIGN
    assert f(A, A, A, A, 7, 1, 4096, 14336, A, None, None) == DTYPE
    assert ts.ffn_workspace_bytes(4, 4096, 14336, 1) <= ts.NOALLOC_SCRATCH_BYTES
    assert ts.ffn_workspace_bytes(8, 4096, 14336, 1) > ts.NOALLOC_SCRATCH_BYTES
