"""bench.py's command-line contract, checked on the CPU: one GPU only, and
default step counts that keep a default run within minutes."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, BENCH, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_defaults():
    spec = importlib.util.spec_from_file_location("bench_contract", BENCH)
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    argv, sys.argv = sys.argv, [BENCH]
    try:
        args = bench.parse()
    finally:
        sys.argv = argv
    assert (args.gpus, args.steps, args.warmup) == (1, 200, 10)
    assert set(args.legs.split(",")) >= {"decode", "prefill", "talker", "restore"}
