"""Host-side launch planner (HIP-free unit ts_plan.cpp): its invariants over
a grid of shapes, slot counts and tuning values, built with g++ and the
address / undefined-behaviour sanitizers."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2406_05955_amd", "csrc")


def test_plan_invariants(tmp_path):
    exe = tmp_path / "plan_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                    os.path.join(ROOT, "tests", "native", "plan_check.cpp"), os.path.join(CSRC, "ts_plan.cpp"),
                    "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


def test_select_key_and_digit_schedule(tmp_path):
    """The top-k selection's key (fp32 bits of the magnitude, sign bit
    cleared, NaN clamped, plus one) and its radix digits (bits 30..23, then
    22..15, 14..7, 7..0): a host model of the selection steps over these
    shared constexpr definitions keeps exactly what a sort keeps, on values
    with signs, ties, infinities and NaN patterns."""
    exe = tmp_path / "select_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                    os.path.join(ROOT, "tests", "native", "select_check.cpp"), "-o", str(exe)], check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr


def test_oracle_under_sanitizers(tmp_path):
    """oracle.c built with the address and undefined-behaviour sanitizers
    (OpenMP on, 1 and 3 threads), every function driven on small fp32 and
    bf16 inputs; exact agreements between functions checked on the way."""
    exe = tmp_path / "oracle_check"
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fopenmp", "-ffp-contract=off",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    os.path.join(ROOT, "tests", "native", "oracle_check.c"), os.path.join(ROOT, "oracle", "oracle.c"),
                    "-lm", "-o", str(exe)], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and r.stdout.strip() == "ok", r.stdout + r.stderr
