"""Concurrent calls: the library keeps no device state between calls, so
calls on two streams with distinct workspaces, enqueued interleaved and
left to overlap, give the same bits as the same calls made one after the
other (single-token, batched and MoE entry points)."""
import numpy as np
import pytest
import torch

from gpu_util import DEV, to_dev
from paper_2406_05955_amd import synth

pytestmark = pytest.mark.gpu

ts = pytest.importorskip("paper_2406_05955_amd.binding") if torch.cuda.is_available() else None


def _inputs(B, H, I, seed):
    inp = synth.make_ffn(B, H, I, gate_bias=-0.84, dtype=synth.BF16, seed=seed)
    return to_dev(inp.x), [to_dev(a) for a in (inp.w_gate, inp.w_up, inp.w_down_t)]


@pytest.mark.parametrize("B", [1, 8])
def test_two_streams_match_serial(B):
    H, I = 2048, 6000
    calls = []
    for k in range(4):
        x, (wg, wu, wd) = _inputs(B, H, I, [70, B, k])
        ws = torch.empty(ts.ffn_workspace_bytes(B, H, I, ts.TS_BF16), dtype=torch.uint8, device=DEV)
        out = torch.empty(B, H, dtype=torch.float32, device=DEV)
        calls.append((x, wg, wu, wd, ws, out))
    serial = []
    for x, wg, wu, wd, ws, out in calls:
        serial.append(ts.ffn_sparse(x, wg, wu, wd, ws=ws).clone())
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for rep in range(3):
        for k, (x, wg, wu, wd, ws, out) in enumerate(calls):
            s = streams[k % 2]
            with torch.cuda.stream(s):
                ts.ffn_sparse(x, wg, wu, wd, out=out, ws=ws, stream=s)
        torch.cuda.synchronize()
        for k, (_, _, _, _, _, out) in enumerate(calls):
            assert torch.equal(out.view(torch.int32), serial[k].view(torch.int32)), (rep, k)


def test_two_streams_moe():
    B, H, I, E, K = 16, 512, 700, 8, 2
    runs = []
    for k in range(2):
        m = synth.make_moe(B, H, I, E, K, gate_bias=-1.5548, dtype=synth.BF16, seed=[71, k])
        args = [to_dev(a) for a in (m.x, m.w_router, m.w_gate, m.w_up, m.w_down_t)]
        ws = torch.empty(ts.moe_workspace_bytes(B, H, I, E, K, ts.TS_BF16), dtype=torch.uint8, device=DEV)
        runs.append((args, ws))
    serial = [ts.moe_sparse(*a, K, ws=ws)[0].clone() for a, ws in runs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    outs = []
    for (a, ws), s in zip(runs, streams):
        with torch.cuda.stream(s):
            outs.append(ts.moe_sparse(*a, K, ws=ws, stream=s)[0])
    torch.cuda.synchronize()
    for got, want in zip(outs, serial):
        assert torch.equal(got.view(torch.int32), want.view(torch.int32))
