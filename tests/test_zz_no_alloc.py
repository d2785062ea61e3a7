"""The allocation-free entry point ts_ffn_sparse_noalloc, called through the
C ABI: it runs ts_ffn_sparse's kernels on the library's fixed scratch array
instead of a caller workspace, so its results must equal ts_ffn_sparse's bit
for bit, and match the fp64 oracle to the same bounds.  Two calls in a row,
the second with a smaller input (another kernel sequence, on the scratch the
first call left behind); a shape whose workspace exceeds the array is
rejected before anything is enqueued and leaves the output untouched."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import DEV, check_ffn_output, ffn_inputs_to_dev, rel_l2
from paper_2406_05955_amd import synth

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2406_05955_amd.binding") if torch.cuda.is_available() else None


def _mistral_layer(seed):
    L = synth.make_ffn_stack_torch(1, 1, 4096, 14336, gate_bias=-0.8416, dtype=synth.BF16, seed=seed, device=DEV)
    h = lambda t: synth.tensor_to_host_array(t, synth.BF16)  # noqa: E731
    return synth.FFNInputs(x=L["x"][0].cpu().numpy(), w_gate=h(L["w_gate"][0]), w_up=h(L["w_up"][0]),
                           w_down_t=h(L["w_down_t"][0]), dtype=synth.BF16, gate_bias=-0.8416)


def _same_as_workspace_path(inp):
    B, H, I = inp.shape
    assert ts.ffn_workspace_bytes(B, H, I, inp.dtype) <= ts.NOALLOC_SCRATCH_BYTES
    ref = oracle.ffn(inp.x, inp.w_gate, inp.w_up, inp.w_down_t, inp.dtype)
    x, wg, wu, wd = ffn_inputs_to_dev(inp)
    a, sa = ts.ffn_sparse(x, wg, wu, wd, stats=True, union=B > 1)
    out = torch.full((B, H), float("nan"), dtype=torch.float32, device=DEV)
    b, sb = ts.ffn_sparse_noalloc(x, wg, wu, wd, out=out, stats=True, union=B > 1)
    torch.cuda.synchronize()
    assert b.data_ptr() == out.data_ptr()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32)), (B, H, I)
    for k in sa:
        if k in ("gate_idx", "active_idx"):
            for t in range(B):
                n = int(sa["n_gate" if k == "gate_idx" else "n_active"][t])
                assert torch.equal(sa[k][t, :n], sb[k][t, :n]), (k, t)
        else:
            assert torch.equal(sa[k], sb[k]), k
    got = b.cpu().numpy()
    assert rel_l2(got, ref.y) <= (1e-5 if inp.dtype == synth.F32 else 1e-2)
    check_ffn_output(got, ref.y, inp.x, inp.w_gate, inp.w_up, inp.w_down_t, ref.g, ref.u,
                     batched=B > 1 and inp.dtype == synth.BF16, what=f"noalloc B={B} H={H} I={I}")


def test_noalloc_two_calls_second_smaller():
    """The Mistral-shaped layer (batch 1, bf16), then a smaller one (two
    tokens: the matrix-core path, another scratch layout), then an fp32
    layer: each equals the workspace entry point's result bit for bit."""
    _same_as_workspace_path(_mistral_layer(seed=90))
    _same_as_workspace_path(synth.make_ffn(2, 1024, 3000, gate_bias=-0.84, dtype=synth.BF16, seed=91))
    _same_as_workspace_path(synth.make_ffn(1, 512, 1792, gate_bias=-0.84, dtype=synth.F32, seed=0))


def test_noalloc_rejects_shapes_beyond_the_scratch():
    """Batch 8 at hidden 4096, inter 14336, bf16 needs about 33 MiB of
    workspace, more than the 32 MiB array: TS_ERR_WORKSPACE, a message
    naming both sizes, nothing enqueued, the output untouched."""
    B, H, I = 8, 4096, 14336
    assert ts.ffn_workspace_bytes(B, H, I, ts.TS_BF16) > ts.NOALLOC_SCRATCH_BYTES
    x = torch.randn(B, H, device=DEV)
    w = torch.zeros(I, H, dtype=torch.bfloat16, device=DEV)
    out = torch.full((B, H), 7.0, device=DEV)
    with pytest.raises(ts.TSError) as e:
        ts.ffn_sparse_noalloc(x, w, w, w, out=out)
    torch.cuda.synchronize()
    assert e.value.code == 5 and "bytes of scratch" in str(e.value)
    assert torch.all(out == 7.0).item()
    # the entry point still serves a fitting shape afterwards
    _same_as_workspace_path(synth.make_ffn(3, 256, 700, gate_bias=-0.5, dtype=synth.BF16, seed=92))


@pytest.mark.parametrize("B", [1, 4])
def test_noalloc_graph_capture(B):
    """What the entry point is for: a call captured into a HIP graph with no
    workspace to allocate.  The first call on the device (warm-up, outside
    the capture) looks the scratch up; the captured call only enqueues
    kernels.  Four replays with new inputs written between them (eager work
    on the same stream), each equal bit for bit to an eager call."""
    from test_gpu_graph import _ffn, replay_check
    H, I = 1024, 2000
    x, (wg, wu, wd), fresh = _ffn(B, H, I, 94)
    out = torch.empty(B, H, dtype=torch.float32, device=DEV)
    replay_check(lambda xx: ts.ffn_sparse_noalloc(xx, wg, wu, wd, out=out if xx is x else None), x, fresh)
