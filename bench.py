#!/usr/bin/env python3
"""Decode-time benchmark of the activation-sparse dReLU FFN on one MI355X.

Default workload: a Mistral-7B-shaped FFN stack (32 independent layers,
hidden 4096, inter 14336, bf16 weights, fp32 accumulation, batch 1), gate
bias column set for ~90% zero Combined activations.  One step is one decode
token through the 32 layers (ts_ffn_sparse per layer: gate + ReLU +
compaction, gathered up, down axpy, cross-block reduction).  Weights are drawn
on the device with a seeded generator and stay resident in HBM; the 32-layer
stack (4.9 GB touched per step) is far larger than the 256 MB last-level cache,
so every step streams its weights from HBM.

Prints one JSON line: tokens/s/layer = batch * layers / (seconds per step),
the dense comparator (ts_ffn_dense) on the same stack, the roofline of the
dominant kernel (ffn_main, the pipelined single-token kernel) from
per-launch HIP events (and, when the committed rocprofv3 trace summary was
taken on the current kernel source, from the trace as well), the fp64 oracle
timed on the host cores as a CPU baseline, and under "configs" every other
workload configuration with its own parity against the oracle: the small
fp32 layer, batch 8 and 32, the MoE layer at batch 1 and 16, and the
50-99% sparsity sweep (shorter runs: --config-steps).

Other workloads (--workload, one JSON line each): sweep (gate bias for
50/75/90/95/99% sparsity), moe (Mixtral-shaped top-2 MoE layer, batch 1, 16,
32, 64), batch (batch 8 and 32), given (predictor mode: each layer called
with its exact gate set as the neuron list), act (dReLU beside ReGLU and the
shifted gate-only ReLU), topk (the top-k magnitude mask).
"""
from __future__ import annotations

import argparse
import ctypes
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
H_MISTRAL, I_MISTRAL = 4096, 14336
# Every source the library is built from: a profile summary stamped with
# another hash was taken on other code, whichever kernel changed.
KERNEL_SOURCES = sorted(
    os.path.relpath(p, ROOT)
    for ext in ("*.hip", "*.h", "*.cpp")
    for p in glob.glob(os.path.join(ROOT, "paper_2406_05955_amd", "csrc", ext))) + [
        "paper_2406_05955_amd/build.py", "include/turbosparse.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_ffn_main_mistral_b1.txt")
TRACE_FILE = os.path.join(ROOT, "profiles", "trace_ffn_main_mistral_b1.txt")


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layers", type=int, default=32)
    ap.add_argument("--workload", default="mistral",
                    choices=["mistral", "sweep", "moe", "batch", "given", "act", "topk", "all"])
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="budget of the oracle CPU-baseline leg")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true")
    ap.add_argument("--probe", action="store_true", help="also run the HBM read / copy probes")
    ap.add_argument("--tile", type=int, default=0, help="ffn_tile tuning knob (0 = default)")
    ap.add_argument("--tune", default="", help="further tuning knobs, KEY=VALUE[,KEY=VALUE...] (ts_tune_set)")
    ap.add_argument("--no-parity", action="store_true", help="skip the oracle parity of the other workloads")
    ap.add_argument("--no-configs", action="store_true",
                    help="default workload: skip the other configurations (small fp32 layer, batch, MoE, sweep)")
    ap.add_argument("--config-steps", type=int, default=10, help="timed steps of each other configuration")
    ap.add_argument("--config-warmup", type=int, default=3, help="warm-up steps of each other configuration")
    ap.add_argument("--batch-sizes", default="8,32", help="batch workload: batch sizes")
    ap.add_argument("--variants", default="independent,hot_cold", help="batch workload: token generators")
    ap.add_argument("--moe-batches", default="1,16,32,64", help="moe workload: batch sizes")
    return ap.parse_args()


def kernel_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_summary(path):
    """The `key: value` lines of a committed profile summary, or None if it
    is missing or was taken on a different kernel source."""
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_hash():
        return None
    return kv


def read_traffic():
    """HBM bytes per launch of ffn_main from the committed counter summary,
    or None if it is missing or was taken on a different kernel source."""
    kv = read_summary(TRAFFIC_FILE)
    try:
        return float(kv["hbm_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def read_trace():
    """ffn_main's average launch duration (us) in the committed rocprofv3
    kernel trace of this benchmark, or None (missing, other source)."""
    kv = read_summary(TRACE_FILE)
    try:
        return (float(kv["ffn_main_avg_us"]), float(kv["ffn_reduce_avg_us"])) if kv else None
    except (KeyError, ValueError):
        return None


class Stack:
    """Device-resident FFN layers and pre-marshalled C-ABI argument tuples."""

    def __init__(self, ts, synth, layers, batch, hidden, inter, gate_bias, seed=0, dtype=None):
        import torch
        self.ts, self.torch, self.synth = ts, torch, synth
        self.dtype = synth.BF16 if dtype is None else dtype
        self.esz = 2 if self.dtype == synth.BF16 else 4
        self.L, self.B, self.H, self.I = layers, batch, hidden, inter
        self.data = synth.make_ffn_stack_torch(layers, batch, hidden, inter, gate_bias=gate_bias,
                                               dtype=self.dtype, seed=seed, device="cuda")
        self.out = torch.empty(layers, batch, hidden, dtype=torch.float32, device="cuda")
        self.wsb = ts.ffn_workspace_bytes(batch, hidden, inter, self.dtype)
        self.ws = torch.empty(self.wsb, dtype=torch.uint8, device="cuda")
        self.stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        vp = ctypes.c_void_p
        self.args = []
        for l in range(layers):
            d = self.data
            self.args.append((vp(d["x"][l].data_ptr()), vp(d["w_gate"][l].data_ptr()), vp(d["w_up"][l].data_ptr()),
                              vp(d["w_down_t"][l].data_ptr()), self.dtype, batch, hidden, inter,
                              vp(self.out[l].data_ptr())))

    def step_sparse(self):
        f = self.ts.lib.ts_ffn_sparse
        for a in self.args:
            rc = f(*a, None, self.ws.data_ptr(), self.wsb, self.stream)
            if rc:
                raise RuntimeError(f"ts_ffn_sparse -> {rc}")

    def step_dense(self):
        f = self.ts.lib.ts_ffn_dense
        for a in self.args:
            rc = f(*a, self.ws.data_ptr(), self.wsb, self.stream)
            if rc:
                raise RuntimeError(f"ts_ffn_dense -> {rc}")

    def counts(self):
        """Per-layer (n_gate, n_active) summed over the batch, and the unions."""
        res = []
        for l in range(self.L):
            d = self.data
            _, st = self.ts.ffn_sparse(d["x"][l], d["w_gate"][l], d["w_up"][l], d["w_down_t"][l], stats=True,
                                       union=self.B > 1)
            self.torch.cuda.synchronize()
            if self.B > 1:
                ng, na = (int(v) for v in st["n_union"].cpu().tolist())
            else:
                ng, na = int(st["n_gate"].sum()), int(st["n_active"].sum())
            res.append((ng, na))
        return res


def timed(torch, fn, steps, warmup):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def kernel_avg_ms(ts, torch, fn, steps, kernel):
    ts.prof_reset()
    ts.prof_enable(True)
    try:
        for _ in range(steps):
            fn()
        torch.cuda.synchronize()
        n, ms = ts.prof_read(kernel)
    finally:
        ts.prof_enable(False)
        ts.prof_reset()
    return n, ms / max(n, 1)


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _layer_host(stack, synth, l):
    d = stack.data
    x = d["x"][l].cpu().numpy()
    w = [synth.tensor_to_host_array(d[k][l], stack.dtype) for k in ("w_gate", "w_up", "w_down_t")]
    return x, w


def _rel_l2(got, want) -> float:
    import numpy as np
    got = np.asarray(got, np.float64)
    n = float(np.linalg.norm(want))
    return float(np.linalg.norm(got - want) / n) if n > 0 else float(np.abs(got).max())


def parity_layers(ts, torch, stack, synth, layers):
    """The sparse path's output of the given stack layers, recomputed into
    fresh buffers, against the fp64 oracle (relative L2 per layer)."""
    import oracle
    d = stack.data
    rel = {}
    for l in layers:
        out = ts.ffn_sparse(d["x"][l], d["w_gate"][l], d["w_up"][l], d["w_down_t"][l])
        torch.cuda.synchronize()
        x, (wg, wu, wd) = _layer_host(stack, synth, l)
        ref = oracle.ffn(x, wg, wu, wd, stack.dtype, threads=oracle.max_threads())
        rel[l] = _rel_l2(out.cpu().numpy(), ref.y)
    return rel


def cpu_baseline(stack, synth, budget_s):
    """The fp64 oracle (test infrastructure) on layer 0 of the stack, on the
    host cores, repeated until the time budget is spent; then a short run on
    one thread."""
    import oracle
    x, (wg, wu, wd) = _layer_host(stack, synth, 0)
    threads = oracle.max_threads()

    def rate(nthreads, budget):
        runs, t0 = 0, time.perf_counter()
        while True:
            oracle.ffn(x, wg, wu, wd, synth.BF16, threads=nthreads)
            runs += 1
            el = time.perf_counter() - t0
            if el >= budget or runs >= 5000:
                return runs, el
    runs, el = rate(threads, budget_s)
    runs1, el1 = rate(1, min(3.0, budget_s))
    return {"value": stack.B * runs / el, "unit": "tokens/s/layer", "cores": threads, "kind": "oracle",
            "sample": f"layer 0 of the stack (H={stack.H}, I={stack.I}, bf16, batch {stack.B}), dense fp64, "
                      f"{runs} runs in {el:.1f} s",
            "value_1_thread": stack.B * runs1 / el1, "cpu_model": _cpu_model()}


def achievable_read(ts, torch, tensors):
    """Read bandwidth of the read probe streaming each tensor once per launch,
    over the list (GB/s): the rate a single launch of that size reaches."""
    sink = torch.empty(4096, dtype=torch.float32, device="cuda")

    def sweep():
        for t in tensors:
            ts.probe_read(t, sink)
    sweep()
    torch.cuda.synchronize()
    n, ms = kernel_avg_ms(ts, torch, sweep, 2, "probe_read")
    return tensors[0].numel() * tensors[0].element_size() / (ms * 1e-3) / 1e9


def bytes_sparse(esz, H, I, ng, na, B):
    return esz * H * (I + ng + na) + 4 * B * H


def roofline_main(ts, torch, stack, counts, steps):
    """Per-kernel HIP-event durations of the single-token path and the
    algorithmic bytes the dominant kernel moves per launch: ffn_main reads
    W_gate whole, the open-gate rows of W_up and the active rows of W_down_t
    (and x).  The partial rows it writes for the cross-block reduction are
    overhead, not algorithmic bytes."""
    H, I, B, L = stack.H, stack.I, stack.B, stack.L
    n_m, m_ms = kernel_avg_ms(ts, torch, stack.step_sparse, steps, "ffn_main")
    n_r, r_ms = kernel_avg_ms(ts, torch, stack.step_sparse, steps, "ffn_reduce")
    alg = sum(bytes_sparse(stack.esz, H, I, ng, na, B) for ng, na in counts) / L
    if n_m == 0 or m_ms <= 0:
        # another kernel sequence (tuning knobs, rows too wide for the
        # pipelined kernel): no ffn_main launch to divide by
        return {"bound": "hbm", "achieved": None, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": None,
                "traffic": None, "kernel": "ffn_main", "launches": 0, "algorithmic_bytes_per_launch": alg,
                "note": "no ffn_main launch recorded in this kernel sequence"}
    ach = alg / (m_ms * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBPS,
            "traffic": read_traffic(), "kernel": "ffn_main", "avg_launch_us": m_ms * 1e3, "launches": n_m,
            "algorithmic_bytes_per_launch": alg,
            "reduce": {"kernel": "ffn_reduce", "avg_launch_us": r_ms * 1e3, "launches": n_r}}


def run_mistral(args, ts, synth, torch):
    B, H, I, L = 1, H_MISTRAL, I_MISTRAL, args.layers
    stack = Stack(ts, synth, L, B, H, I, gate_bias=-0.8416)
    # correctness-side pass (not timed): per-layer active counts for the byte model
    counts = stack.counts()
    t_sparse = timed(torch, stack.step_sparse, args.steps, args.warmup)
    esz = 2
    per_layer = [bytes_sparse(esz, H, I, ng, na, B) for ng, na in counts]
    alg_bytes = sum(per_layer) / L
    dense_bytes = 3 * esz * H * I + 4 * B * H
    res = {
        "metric": "sparse-FFN decode tokens/s/layer + achieved HBM GB/s vs dense GEMV",
        "value": B * L / t_sparse,
        "unit": "tokens/s/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_sparse * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded device RNG; random weights of the Mistral-7B FFN shape)",
        "config": {"workload": "mistral7b_ffn_stack_bf16_b1_s90", "layers": L, "batch": B, "hidden": H,
                   "inter": I, "combined_sparsity_target": 0.90,
                   "measured_gate_fraction": sum(c[0] for c in counts) / (L * I),
                   "measured_combined_sparsity": 1 - sum(c[1] for c in counts) / (L * I)},
        "hbm_GBps_touched": alg_bytes / (t_sparse / L) / 1e9,
        "hbm_frac_touched": alg_bytes / (t_sparse / L) / 1e9 / HBM_PEAK_GBPS,
        "touched_bytes_per_layer": alg_bytes,
        "roofline": roofline_main(ts, torch, stack, counts, args.steps),
    }
    # the measured ceiling for a launch of this size: the read probe streaming
    # one layer's W_gate (117 MB) per launch, over the stack's layers
    ach_read = achievable_read(ts, torch, list(stack.data["w_gate"]))
    res["roofline"]["achievable_GBps"] = ach_read
    if res["roofline"]["achieved"]:
        res["roofline"]["frac_of_achievable"] = res["roofline"]["achieved"] / ach_read
    tr = read_trace()
    if tr:
        # the same kernel's duration in the committed rocprofv3 trace of this
        # benchmark (same source): a second clock for the same quantity
        res["roofline"]["trace"] = {"avg_launch_us": tr[0], "achieved": alg_bytes / (tr[0] * 1e-6) / 1e9,
                                    "frac": alg_bytes / (tr[0] * 1e-6) / 1e9 / HBM_PEAK_GBPS,
                                    "reduce_avg_launch_us": tr[1],
                                    "source": os.path.relpath(TRACE_FILE, ROOT)}
    res["roofline"]["achievable_probe"] = (f"probe_read streaming one layer's W_gate "
                                           f"({stack.data['w_gate'][0].numel() * 2 / 1e6:.1f} MB) per launch, "
                                           f"{L} layers")
    if not args.no_dense:
        t_dense = timed(torch, stack.step_dense, args.steps, args.warmup)
        res["dense"] = {"value": B * L / t_dense, "unit": "tokens/s/layer", "ms_per_step": t_dense * 1e3,
                        "hbm_GBps_touched": dense_bytes / (t_dense / L) / 1e9,
                        "speedup_sparse_vs_dense": t_dense / t_sparse,
                        "byte_bound_speedup": dense_bytes / alg_bytes}
    if args.probe:
        res["probe"] = run_probes(ts, torch)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(stack, synth, args.cpu_seconds)
        rel = parity_layers(ts, torch, stack, synth, (0, L - 1))
        res["parity_layer0_rel_l2"] = rel[0]
        res["parity_last_layer_rel_l2"] = rel[L - 1]
    if not args.no_configs:
        res["configs"] = run_configs(args, ts, synth, torch)
    res["paper_context"] = {
        "note": "context only: other hardware, whole-model decode, predictor-driven PowerInfer vs dense llama.cpp",
        "decode_speedup": "2-5x (i9-14900HX + RTX 4090 Laptop; i7-12700K + RTX 2080Ti)",
        "phone": "11.1 tokens/s TurboSparse-Mixtral-47B INT4, OnePlus-12 (Snapdragon 8 Gen 3), llama.cpp 0.5"}
    res["kernel_source_sha256_16"] = kernel_hash()
    return res


def run_probes(ts, torch):
    nbytes = 4 << 30
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").normal_()
    sink = torch.empty(4096, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src[: (256 << 20) // 2])
    for _ in range(2):
        ts.probe_read(src, sink)
        ts.probe_copy(src[: dst.numel()], dst)
    torch.cuda.synchronize()
    n, ms = kernel_avg_ms(ts, torch, lambda: ts.probe_read(src, sink), 5, "probe_read")
    n2, ms2 = kernel_avg_ms(ts, torch, lambda: ts.probe_copy(src[: dst.numel()], dst), 5, "probe_copy")
    return {"read_GBps": nbytes / (ms * 1e-3) / 1e9, "read_bytes": nbytes,
            "copy_GBps": 2 * dst.numel() * 2 / (ms2 * 1e-3) / 1e9, "copy_bytes": dst.numel() * 2}


SWEEP = (0.50, 0.75, 0.90, 0.95, 0.99)


def ffn_entry(args, ts, synth, torch, workload, batch, gate_bias, seed, dtype=None, hidden=H_MISTRAL,
              inter=I_MISTRAL, layers=None, steps=None, warmup=None, parity=True, extra=None):
    """One FFN stack configuration, measured: tokens/s/layer and touched
    GB/s of the sparse path, the dense comparator on the same stack, the
    byte-bound speedup, the dominant kernels' event-pair durations, and the
    parity of the first and last layers against the fp64 oracle."""
    L = layers or args.layers
    steps = steps or args.steps
    warmup = args.warmup if warmup is None else warmup
    stack = Stack(ts, synth, L, batch, hidden, inter, gate_bias=gate_bias, seed=seed, dtype=dtype)
    counts = stack.counts()  # per layer (n_G, n_A); unions over the batch when batch > 1
    H, I, B, esz = hidden, inter, batch, stack.esz
    t_s = timed(torch, stack.step_sparse, steps, warmup)
    t_d = None if args.no_dense else timed(torch, stack.step_dense, steps, warmup)
    alg = sum(bytes_sparse(esz, H, I, ng, na, B) for ng, na in counts) / L
    dense = 3 * esz * H * I + 4 * B * H
    res = {"workload": workload, "batch": B, "hidden": H, "inter": I, "layers": L,
           "dtype": "bf16" if stack.dtype == synth.BF16 else "f32", "steps": steps, **(extra or {}),
           ("union_gate_fraction" if B > 1 else "gate_fraction"): sum(c[0] for c in counts) / (L * I),
           ("union_active_fraction" if B > 1 else "active_fraction"): sum(c[1] for c in counts) / (L * I),
           "us_per_layer": t_s / L * 1e6, "sparse_tokens_per_s_layer": B * L / t_s,
           "touched_bytes_per_layer": alg, "sparse_GBps_touched": alg / (t_s / L) / 1e9,
           "sparse_frac_touched": alg / (t_s / L) / 1e9 / HBM_PEAK_GBPS}
    if t_d:
        res.update({"dense_tokens_per_s_layer": B * L / t_d, "dense_GBps": dense / (t_d / L) / 1e9,
                    "speedup_vs_dense": t_d / t_s, "byte_bound_speedup": dense / alg,
                    "target_speedup_0.6x_byte_bound": 0.6 * dense / alg})
    kst = max(3, steps // 2)
    if B == 1 or stack.dtype != synth.BF16:
        rl = roofline_main(ts, torch, stack, counts, kst)
        res.update({"ffn_main_us": rl.get("avg_launch_us"), "ffn_main_GBps": rl.get("achieved"),
                    "ffn_main_frac": rl.get("frac"),
                    "ffn_reduce_us": rl.get("reduce", {}).get("avg_launch_us")})
    else:
        kt = batch_kernels(ts, torch, stack.step_sparse, kst)
        res.update(kt)
        gu = sum(esz * H * (I + ng) for ng, _ in counts) / L
        dn = sum(esz * H * na for _, na in counts) / L
        res["gate_up_bytes_per_layer"], res["down_bytes_per_layer"] = gu, dn
        if kt.get("batch_gate_up_us"):
            res["batch_gate_up_GBps"] = gu / (kt["batch_gate_up_us"] * 1e-6) / 1e9
        if kt.get("batch_down_us"):
            res["batch_down_GBps"] = dn / (kt["batch_down_us"] * 1e-6) / 1e9
    if parity and not args.no_parity:
        rel = parity_layers(ts, torch, stack, synth, (0, L - 1))
        res["parity_layer0_rel_l2"] = rel[0]
        res["parity_last_layer_rel_l2"] = rel[L - 1]
    del stack
    torch.cuda.empty_cache()
    return res


def run_sweep(args, ts, synth, torch):
    """Gate bias set for 50/75/90/95/99% zero Combined activations on the
    Mistral-shaped stack, batch 1; dense comparator on every point."""
    out = []
    for s in SWEEP:
        b = synth.gate_bias_for_combined_sparsity(s)
        out.append(ffn_entry(args, ts, synth, torch, f"mistral7b_ffn_stack_bf16_b1_s{round(s * 100)}", 1, b, seed=1,
                             extra={"target_sparsity": s, "gate_bias": b,
                                    "literal_target_0.6_over_1_minus_s": 0.6 / (1 - s)}))
    return out


def run_given_workload(args, ts, synth, torch):
    """Predictor mode on the Mistral-shaped stack, batch 1: each layer is
    called with an externally supplied neuron list (ts_ffn_sparse_given), here
    the exact gate set G of the layer's token (what a perfect activation
    predictor would return), so W_gate is read only for the listed rows.
    Points at 90% and 99% zero Combined activations."""
    out = []
    H, I, L = H_MISTRAL, I_MISTRAL, args.layers
    for s in (0.90, 0.99):
        b = synth.gate_bias_for_combined_sparsity(s)
        stack = Stack(ts, synth, L, 1, H, I, gate_bias=b, seed=3)
        d = stack.data
        lists, counts = [], []
        for l in range(L):
            _, st = ts.ffn_sparse(d["x"][l], d["w_gate"][l], d["w_up"][l], d["w_down_t"][l], stats=True)
            torch.cuda.synchronize()
            ng, na = int(st["n_gate"][0]), int(st["n_active"][0])
            lists.append((st["gate_idx"][:, :max(ng, 1)].contiguous(),
                          torch.tensor([ng], dtype=torch.int32, device="cuda")))
            counts.append((ng, na))
        maxc = max(int(li.shape[1]) for li, _ in lists)
        wsb = ts.ffn_given_workspace_bytes(1, H, I, maxc, ts.TS_BF16)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        f = ts.lib.ts_ffn_sparse_given
        stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        vp = ctypes.c_void_p
        argl = [(vp(d["x"][l].data_ptr()), vp(d["w_gate"][l].data_ptr()), vp(d["w_up"][l].data_ptr()),
                 vp(d["w_down_t"][l].data_ptr()), ts.TS_BF16, 1, H, I, vp(lists[l][0].data_ptr()),
                 vp(lists[l][1].data_ptr()), int(lists[l][0].shape[1]), vp(stack.out[l].data_ptr()))
                for l in range(L)]

        def step_given():
            for a in argl:
                rc = f(*a, None, ws.data_ptr(), wsb, stream)
                if rc:
                    raise RuntimeError(f"ts_ffn_sparse_given -> {rc}")
        tg = timed(torch, step_given, args.steps, args.warmup)
        tsp = timed(torch, stack.step_sparse, args.steps, args.warmup)
        td = timed(torch, stack.step_dense, args.steps, args.warmup)
        n, ms = kernel_avg_ms(ts, torch, step_given, max(3, args.steps // 3), "ffn_given")
        # bytes: W_gate, W_up rows of the listed (= open) neurons, W_down_t rows of A, x and out
        alg = sum(2 * H * (2 * ng + na) + 8 * H for ng, na in counts) / L
        dense = 3 * 2 * H * I + 8 * H
        out.append({"workload": "mistral7b_ffn_stack_bf16_b1_given_gate_set", "target_sparsity": s,
                    "measured_sparsity": 1 - sum(c[1] for c in counts) / (L * I),
                    "given_tokens_per_s_layer": L / tg, "sparse_tokens_per_s_layer": L / tsp,
                    "dense_tokens_per_s_layer": L / td, "speedup_vs_dense": td / tg,
                    "byte_bound_speedup": dense / alg, "literal_target_0.6_over_1_minus_s": 0.6 / (1 - s),
                    "touched_bytes_per_layer": alg, "given_GBps_touched": alg / (tg / L) / 1e9,
                    "ffn_given_us": ms * 1e3 if n else None})
        del stack, lists, ws
        torch.cuda.empty_cache()
    return out


def run_act_workload(args, ts, synth, torch):
    """Activations side by side on the Mistral-shaped stack, batch 1
    (ts_ffn_sparse_act): dReLU and ReGLU at the same gate bias (20% of the
    gates open), and the shifted gate-only ReLU with its threshold set for
    10% open gates (90% zero Combined activations, as dReLU's point)."""
    out = []
    H, I, L = H_MISTRAL, I_MISTRAL, args.layers
    b = -0.8416
    stack = Stack(ts, synth, L, 1, H, I, gate_bias=b, seed=5)
    d = stack.data
    td = timed(torch, stack.step_dense, args.steps, args.warmup)
    f = ts.lib.ts_ffn_sparse_act
    # gate ~ N(b, ~1): P(gate > tau) = 0.1 at tau = b + 1.2816
    for name, act, tau in (("drelu", ts.TS_ACT_DRELU, 0.0), ("reglu", ts.TS_ACT_RELU_GATE, 0.0),
                           ("shifted_relu_gate", ts.TS_ACT_RELU_GATE, b + 1.2816)):
        counts = []
        for l in range(L):
            _, st = ts.ffn_sparse_act(d["x"][l], d["w_gate"][l], d["w_up"][l], d["w_down_t"][l], act, tau,
                                      stats=True)
            torch.cuda.synchronize()
            counts.append((int(st["n_gate"][0]), int(st["n_active"][0])))

        def step():
            for a in stack.args:
                rc = f(*a[:8], act, ctypes.c_float(tau), a[8], None, stack.ws.data_ptr(), stack.wsb, stack.stream)
                if rc:
                    raise RuntimeError(f"ts_ffn_sparse_act -> {rc}")
        t = timed(torch, step, args.steps, args.warmup)
        alg = sum(2 * H * (I + ng + na) + 8 * H for ng, na in counts) / L
        dense = 3 * 2 * H * I + 8 * H
        out.append({"workload": "mistral7b_ffn_stack_bf16_b1_activation", "activation": name, "tau": tau,
                    "gate_fraction": sum(c[0] for c in counts) / (L * I),
                    "active_fraction": sum(c[1] for c in counts) / (L * I),
                    "sparse_tokens_per_s_layer": L / t, "dense_tokens_per_s_layer": L / td,
                    "speedup_vs_dense": td / t, "byte_bound_speedup": dense / alg,
                    "touched_bytes_per_layer": alg, "sparse_GBps_touched": alg / (t / L) / 1e9})
    del stack
    torch.cuda.empty_cache()
    return out


def run_topk_workload(args, ts, synth, torch):
    """The top-k magnitude mask on the Mistral-shaped stack, batch 1
    (ts_ffn_sparse_topk): keep 5% and 10% of the 14336 neurons per token
    (about half, and about all, of dReLU's ~10% non-zero activations)."""
    out = []
    H, I, L = H_MISTRAL, I_MISTRAL, args.layers
    stack = Stack(ts, synth, L, 1, H, I, gate_bias=-0.8416, seed=5)
    d = stack.data
    td = timed(torch, stack.step_dense, args.steps, args.warmup)
    f = ts.lib.ts_ffn_sparse_topk
    for keep in (I // 20, I // 10):
        counts = []
        for l in range(L):
            _, st = ts.ffn_sparse_topk(d["x"][l], d["w_gate"][l], d["w_up"][l], d["w_down_t"][l], keep,
                                       stats=True)
            torch.cuda.synchronize()
            counts.append((int(st["n_gate"][0]), int(st["n_active"][0])))

        def step():
            for a in stack.args:
                rc = f(*a[:8], keep, a[8], None, stack.ws.data_ptr(), stack.wsb, stack.stream)
                if rc:
                    raise RuntimeError(f"ts_ffn_sparse_topk -> {rc}")
        t = timed(torch, step, args.steps, args.warmup)
        kt = {}
        for k in ("ffn_gate_up", "ffn_topk_select", "ffn_down", "ffn_topk_down", "ffn_reduce"):
            n, ms = kernel_avg_ms(ts, torch, step, max(3, args.steps // 3), k)
            if n:
                kt[k + "_us"] = ms * 1e3
        # gate rows whole, up rows of G, down rows of the kept set, x and out
        alg = sum(2 * H * (I + ng + nk) + 8 * H for ng, nk in counts) / L
        dense = 3 * 2 * H * I + 8 * H
        out.append({"workload": "mistral7b_ffn_stack_bf16_b1_topk", "keep": keep,
                    "gate_fraction": sum(c[0] for c in counts) / (L * I),
                    "kept_fraction": sum(c[1] for c in counts) / (L * I),
                    "sparse_tokens_per_s_layer": L / t, "dense_tokens_per_s_layer": L / td,
                    "speedup_vs_dense": td / t, "byte_bound_speedup": dense / alg,
                    "touched_bytes_per_layer": alg, "sparse_GBps_touched": alg / (t / L) / 1e9,
                    "us_per_layer": t / L * 1e6, **kt})
    del stack
    torch.cuda.empty_cache()
    return out


def batch_kernels(ts, torch, fn, steps):
    res = {}
    for k in ("moe_router", "batch_prep", "batch_gate_up", "batch_down", "batch_reduce"):
        n, ms = kernel_avg_ms(ts, torch, fn, steps, k)
        if n:
            res[k + "_us"] = ms * 1e3
    return res


def run_batch_workload(args, ts, synth, torch):
    """Mistral-shaped FFN stack with a batch of independent decode tokens
    (batch 8 and 32): literal generator (each token ~90% sparse, union grows
    with the batch) and the skewed hot/cold variant (union ~67% sparse)."""
    out = []
    for B in (int(b) for b in args.batch_sizes.split(",")):
        for variant in args.variants.split(","):
            bias = -0.8416 if variant == "independent" else synth.hot_cold_bias(I_MISTRAL, seed=11)
            out.append(ffn_entry(args, ts, synth, torch, f"mistral7b_ffn_stack_bf16_b{B}_{variant}", B, bias, seed=2,
                                 extra={"variant": variant}))
    return out


class MoEStack:
    """Device-resident MoE layers (router + packed experts) and marshalled
    C-ABI arguments."""

    def __init__(self, ts, synth, layers, batch, hidden, inter, E, K, gate_bias, seed=0):
        import torch
        self.ts, self.torch = ts, torch
        self.L, self.B, self.H, self.I, self.E, self.K = layers, batch, hidden, inter, E, K
        self.d = synth.make_moe_stack_torch(layers, batch, hidden, inter, E, K, gate_bias=gate_bias,
                                            dtype=synth.BF16, seed=seed, device="cuda")
        self.out = torch.empty(layers, batch, hidden, dtype=torch.float32, device="cuda")
        self.idx = torch.empty(layers, batch, K, dtype=torch.int32, device="cuda")
        self.w = torch.empty(layers, batch, K, dtype=torch.float32, device="cuda")
        self.wsb = ts.moe_workspace_bytes(batch, hidden, inter, E, K, ts.TS_BF16)
        self.ws = torch.empty(self.wsb, dtype=torch.uint8, device="cuda")
        self.stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        vp = ctypes.c_void_p
        self.args = [(vp(self.d["x"][l].data_ptr()), vp(self.d["w_router"][l].data_ptr()),
                      vp(self.d["w_gate"][l].data_ptr()), vp(self.d["w_up"][l].data_ptr()),
                      vp(self.d["w_down_t"][l].data_ptr()), ts.TS_BF16, batch, hidden, inter, E, K,
                      vp(self.out[l].data_ptr()), vp(self.idx[l].data_ptr()), vp(self.w[l].data_ptr()))
                     for l in range(layers)]

    def step_sparse(self):
        f = self.ts.lib.ts_moe_sparse
        for a in self.args:
            rc = f(*a, None, self.ws.data_ptr(), self.wsb, self.stream)
            if rc:
                raise RuntimeError(f"ts_moe_sparse -> {rc}")

    def step_dense(self):
        f = self.ts.lib.ts_moe_dense
        for a in self.args:
            rc = f(*a, self.ws.data_ptr(), self.wsb, self.stream)
            if rc:
                raise RuntimeError(f"ts_moe_dense -> {rc}")

    def touched(self):
        """Per layer: algorithmic bytes of the sparse MoE (router, and for each
        expert hit its whole W_gate plus the union rows of W_up / W_down_t
        over the tokens routed to it) and of the dense-routed comparator."""
        import numpy as np
        sp, dn = [], []
        H, I, B, K = self.H, self.I, self.B, self.K
        for l in range(self.L):
            d = self.d
            _, idx, _, st = self.ts.moe_sparse(d["x"][l], d["w_router"][l], d["w_gate"][l], d["w_up"][l],
                                               d["w_down_t"][l], K, stats=True)
            self.torch.cuda.synchronize()
            idx = idx.cpu().numpy()
            ng, na = st["n_gate"].cpu().numpy(), st["n_active"].cpu().numpy()
            gi, ai = st["gate_idx"].cpu().numpy(), st["active_idx"].cpu().numpy()
            b = 2 * self.E * H + 8 * B * H
            bd = b
            for e in np.unique(idx):
                gsets, asets = [], []
                for t in range(B):
                    for k in range(K):
                        if idx[t, k] == e:
                            s = t * K + k
                            gsets.append(gi[s, :ng[s]])
                            asets.append(ai[s, :na[s]])
                ug = len(np.unique(np.concatenate(gsets))) if gsets else 0
                ua = len(np.unique(np.concatenate(asets))) if asets else 0
                b += 2 * H * (I + ug + ua)
                bd += 3 * 2 * H * I
            sp.append(b)
            dn.append(bd)
        return sp, dn


def parity_moe_layers(ts, torch, stack, synth, layers):
    """The sparse MoE layer's output of the given stack layers against the
    fp64 oracle (relative L2 over the tokens whose k-th and (k+1)-th oracle
    probabilities are not within 1e-6, relative; routing compared on them)."""
    import numpy as np
    import oracle
    d, K, E = stack.d, stack.K, stack.E
    rel, route_ok = {}, True
    h = lambda t: synth.tensor_to_host_array(t, synth.BF16)  # noqa: E731
    for l in layers:
        out, idx, _ = ts.moe_sparse(d["x"][l], d["w_router"][l], d["w_gate"][l], d["w_up"][l], d["w_down_t"][l], K)
        torch.cuda.synchronize()
        ref = oracle.moe(d["x"][l].cpu().numpy(), h(d["w_router"][l]), h(d["w_gate"][l]), h(d["w_up"][l]),
                         h(d["w_down_t"][l]), synth.BF16, K, threads=oracle.max_threads(), keep_projections=False)
        p = np.sort(ref.probs, axis=1)[:, ::-1]
        keep = [t for t in range(stack.B) if not (K < E and abs(p[t, K - 1] - p[t, K]) <= 1e-6 * p[t, K - 1])]
        rel[l] = _rel_l2(out.cpu().numpy()[keep], ref.y[keep])
        route_ok = route_ok and idx.cpu().numpy()[keep].tolist() == ref.topk_idx[keep].tolist()
    return rel, route_ok


def moe_entry(args, ts, synth, torch, B, sp_target, bias, layers=8, steps=None, warmup=None, parity=True):
    """Mixtral-shaped MoE layer stack (8 experts, top 2, bf16), measured as
    ffn_entry measures the FFN."""
    H, I, E, K, L = H_MISTRAL, I_MISTRAL, 8, 2, layers
    steps = steps or args.steps
    warmup = args.warmup if warmup is None else warmup
    stack = MoEStack(ts, synth, L, B, H, I, E, K, gate_bias=bias, seed=4)
    sp, dn = stack.touched()
    t_s = timed(torch, stack.step_sparse, steps, warmup)
    t_d = None if args.no_dense else timed(torch, stack.step_dense, steps, warmup)
    alg, dense = sum(sp) / L, sum(dn) / L
    res = {"workload": f"mixtral_moe_bf16_b{B}_s{int(sp_target * 100)}", "batch": B, "layers": L, "experts": E,
           "top_k": K, "in_expert_sparsity_target": sp_target, "gate_bias": bias, "steps": steps,
           "us_per_layer": t_s / L * 1e6, "sparse_tokens_per_s_layer": B * L / t_s,
           "touched_bytes_per_layer": alg, "sparse_GBps_touched": alg / (t_s / L) / 1e9,
           "sparse_frac_touched": alg / (t_s / L) / 1e9 / HBM_PEAK_GBPS}
    if t_d:
        res.update({"dense_tokens_per_s_layer": B * L / t_d, "dense_GBps": dense / (t_d / L) / 1e9,
                    "speedup_vs_dense": t_d / t_s, "byte_bound_speedup": dense / alg,
                    "target_speedup_0.6x_byte_bound": 0.6 * dense / alg})
    kst = max(3, steps // 2)
    if B == 1:
        for k in ("moe_router", "ffn_main", "ffn_reduce"):
            n, ms = kernel_avg_ms(ts, torch, stack.step_sparse, kst, k)
            if n:
                res[k + "_us"] = ms * 1e3
    else:
        res.update(batch_kernels(ts, torch, stack.step_sparse, kst))
    if parity and not args.no_parity:
        rel, route_ok = parity_moe_layers(ts, torch, stack, synth, (0, L - 1))
        res["parity_layer0_rel_l2"] = rel[0]
        res["parity_last_layer_rel_l2"] = rel[L - 1]
        res["parity_routing_exact"] = route_ok
    del stack
    torch.cuda.empty_cache()
    return res


def run_moe_workload(args, ts, synth, torch):
    """Mixtral-shaped MoE layer: 8 experts (hidden 4096, inter 14336, bf16),
    top-2 softmax router, gate bias for 97% zero Combined activations inside
    each expert (also the paper's 85% point at batch 1 and 16), batch 1, 16,
    32 and 64; 8 layers so a step streams several GB."""
    out = []
    for B in (int(b) for b in args.moe_batches.split(",")):
        for sp_target, bias in ((0.97, -1.5548), (0.85, -0.5244)):
            if B > 16 and sp_target == 0.85:
                continue
            out.append(moe_entry(args, ts, synth, torch, B, sp_target, bias))
    return out


def run_configs(args, ts, synth, torch):
    """Every workload configuration besides the headline one, shorter runs
    (args.config_steps timed steps each), keyed by configuration:
    the small fp32 layer (256 copies, so a step streams from HBM), batch 8
    and 32 (independent tokens and the hot/cold variant), the MoE layer at
    batch 1 (97% and 85% in-expert sparsity) and 16, and the sparsity sweep."""
    st, wu = args.config_steps, args.config_warmup
    c = {}
    c["config0_f32_h512_i1792_b1"] = ffn_entry(
        args, ts, synth, torch, "small_ffn_f32_h512_i1792_b1_x256", 1, -0.84, seed=0, dtype=synth.F32, hidden=512,
        inter=1792, layers=256, steps=st, warmup=wu,
        extra={"note": "256 independent copies of the layer so every step streams from HBM"})
    for B in (8, 32):
        for variant in ("independent", "hot_cold"):
            bias = -0.8416 if variant == "independent" else synth.hot_cold_bias(I_MISTRAL, seed=11)
            c[f"config2_b{B}_{variant}"] = ffn_entry(
                args, ts, synth, torch, f"mistral7b_ffn_stack_bf16_b{B}_{variant}", B, bias, seed=2, steps=st,
                warmup=wu, extra={"variant": variant})
    for B, sp_target, bias in ((1, 0.97, -1.5548), (1, 0.85, -0.5244), (16, 0.97, -1.5548), (16, 0.85, -0.5244)):
        c[f"config3_moe_b{B}_s{int(sp_target * 100)}"] = moe_entry(args, ts, synth, torch, B, sp_target, bias,
                                                                    steps=st, warmup=wu)
    for s in SWEEP:
        b = synth.gate_bias_for_combined_sparsity(s)
        c[f"config4_s{round(s * 100)}"] = ffn_entry(
            args, ts, synth, torch, f"mistral7b_ffn_stack_bf16_b1_s{round(s * 100)}", 1, b, seed=1, steps=st,
            warmup=wu, extra={"target_sparsity": s, "gate_bias": b,
                              "literal_target_0.6_over_1_minus_s": 0.6 / (1 - s)})
    return c


def main():
    args = parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1",
                          "n_gpus_requested": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2406_05955_amd import binding as ts
    from paper_2406_05955_amd import synth
    if args.tile:
        ts.tune_set("ffn_tile", args.tile)
    for kv in filter(None, args.tune.split(",")):
        k, v = kv.split("=")
        ts.tune_set(k.strip(), int(v))
    if args.workload == "mistral":
        print(json.dumps(run_mistral(args, ts, synth, torch)), flush=True)
        return
    runs = {"sweep": run_sweep, "batch": run_batch_workload, "moe": run_moe_workload, "given": run_given_workload,
            "act": run_act_workload, "topk": run_topk_workload}
    names = list(runs) if args.workload == "all" else [args.workload]
    for n in names:
        for r in runs[n](args, ts, synth, torch):
            print(json.dumps(r), flush=True)


if __name__ == "__main__":
    main()
