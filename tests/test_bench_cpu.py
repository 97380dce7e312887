"""bench.py's host-side contract (no GPU): more than one GPU is refused with a
message and exit status 2, and the argument parser knows every knob."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args, env=None):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True,
                          text=True, timeout=120, env=env, cwd=ROOT)


def test_more_than_one_gpu_exits_with_message():
    p = run("--gpus", "2")
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_world_size_above_one_exits_with_message():
    env = dict(os.environ, WORLD_SIZE="4")
    p = run(env=env)
    assert p.returncode == 2 and "one GPU" in p.stderr


def test_help_lists_the_knobs():
    p = run("--help")
    assert p.returncode == 0
    for k in ("--steps", "--warmup", "--workload", "--pad-kib", "--priority", "--variant", "--gemm-grid",
              "--comm-wgs", "--comm-rate-gbs", "--cpu-budget", "--no-cpu-baseline"):
        assert k in p.stdout, k
