"""bench.py's host-side logic on the CPU: the one-GPU refusal, the staleness
rule of the committed HBM-traffic summary, and the algorithmic byte count the
roofline divides by."""
import importlib.util
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def load_bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert msg["n_gpus_requested"] == 2 and "one GPU" in msg["error"]


def test_traffic_summary_is_used_only_for_the_source_it_was_taken_on(tmp_path, monkeypatch):
    b = load_bench()
    f = tmp_path / "traffic.txt"
    monkeypatch.setattr(b, "TRAFFIC_FILE", str(f))
    assert b.read_traffic() is None  # missing
    f.write_text(f"# counters\nkernel_source_sha256_16: {b.kernel_hash()}\nhbm_bytes_per_launch: 153290000\n")
    assert b.read_traffic() == 153290000.0
    f.write_text("kernel_source_sha256_16: 0123456789abcdef\nhbm_bytes_per_launch: 153290000\n")
    assert b.read_traffic() is None  # taken on another kernel source
    f.write_text(f"kernel_source_sha256_16: {b.kernel_hash()}\nhbm_bytes_per_launch: n/a\n")
    assert b.read_traffic() is None  # malformed


def test_kernel_hash_covers_the_kernel_sources():
    b = load_bench()
    assert len(b.kernel_hash()) == 16
    for p in b.KERNEL_SOURCES:
        assert os.path.exists(os.path.join(ROOT, p)), p
    for name in ("ts_ffn.hip", "ts_batch.hip", "ts_batch.h", "ts_device.h", "ts_plan.cpp", "ts_plan.h",
                 "ts_runtime.cpp", "ts_probe.hip", "build.py", "turbosparse.h"):
        assert any(p.endswith(name) for p in b.KERNEL_SOURCES), name


def test_algorithmic_bytes():
    """W_gate whole (I rows), the W_up rows of the open gates (|G|), the
    W_down_t rows of the active neurons (|A|), each H elements, plus x in
    fp32: at the Mistral shape with 20% open gates and 10% active, bf16."""
    b = load_bench()
    H, I, ng, na = 4096, 14336, 2867, 1433
    assert b.bytes_sparse(2, H, I, ng, na, 1) == 2 * H * I + 2 * H * ng + 2 * H * na + 4 * H
    assert b.bytes_sparse(4, 8, 10, 0, 0, 3) == 4 * 8 * 10 + 4 * 3 * 8


def test_trace_summary_is_used_only_for_the_source_it_was_taken_on(tmp_path, monkeypatch):
    b = load_bench()
    f = tmp_path / "trace.txt"
    monkeypatch.setattr(b, "TRACE_FILE", str(f))
    assert b.read_trace() is None
    f.write_text(f"kernel_source_sha256_16: {b.kernel_hash()}\nffn_main_avg_us: 27.25\nffn_reduce_avg_us: 4.15\n")
    assert b.read_trace() == (27.25, 4.15)
    f.write_text("kernel_source_sha256_16: 0123456789abcdef\nffn_main_avg_us: 27.25\nffn_reduce_avg_us: 4.15\n")
    assert b.read_trace() is None


def test_roofline_without_main_kernel_launches():
    """A kernel sequence without ffn_main launches (tuning knobs, rows too
    wide for the pipelined kernel) reports a null roofline instead of
    dividing by zero."""
    b = load_bench()

    class FakeTS:
        def prof_reset(self):
            pass

        def prof_enable(self, on):
            pass

        def prof_read(self, kernel):
            return 0, 0.0

    class FakeTorch:
        class cuda:
            @staticmethod
            def synchronize():
                pass

    class FakeStack:
        H, I, B, L, esz = 4096, 14336, 1, 2, 2

        def step_sparse(self):
            pass

    rl = b.roofline_main(FakeTS(), FakeTorch(), FakeStack(), [(2867, 1433), (2867, 1433)], 3)
    assert rl["achieved"] is None and rl["frac"] is None and rl["launches"] == 0
    assert rl["algorithmic_bytes_per_launch"] == b.bytes_sparse(2, 4096, 14336, 2867, 1433, 1)
