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


def test_sweep_table_renders_partial_rows():
    sys.path.insert(0, ROOT)
    from paper_2606_09200_amd import sweep
    rows = [{"workload": "cb", "gemm_variant": 16, "pad_kib": 0, "comm_priority": 0, "t_seq_ms": 10.5,
             "t_ovl_ms": 9.7, "comm_coresident": 0.9},
            {"workload": "sweep", "pad_kib": 128, "comm_priority": 3, "feasible": False}]
    t = sweep.table(rows).splitlines()
    assert len(t) == 4 and t[0].startswith("| workload |")
    ncol = t[0].count("|")
    assert all(line.count("|") == ncol for line in t)
    assert "| 0.900 |" in t[2] and "| 9.7 |" in t[2]


def test_power_sampler_reads_microwatts_per_phase(tmp_path):
    # kernel_driver --sustain --power: samples a hwmon-style file (microwatts)
    # per labelled phase and summarises median and maximum in watts
    import time
    sys.path.insert(0, ROOT)
    from paper_2606_09200_amd import kernel_driver as kd
    f = tmp_path / "power1_input"
    f.write_text("250000000\n")
    s = kd.PowerSampler(str(f))
    s.start()
    time.sleep(0.3)
    s.phase = 0
    f.write_text("1400000000\n")
    time.sleep(0.3)
    s.stop()
    assert s.summary("idle").startswith("median 250 W, max 250 W")
    assert "max 1400 W" in s.summary(0)
    assert s.summary("never") == "no samples"


def test_current_engine_clock_from_a_dpm_listing():
    sys.path.insert(0, ROOT)
    from paper_2606_09200_amd import kernel_driver as kd
    assert kd.current_mhz("S: 102Mhz *\n0: 500Mhz\n1: 2400Mhz\n") == 102.0
    assert kd.current_mhz("0: 500Mhz\n1: 2400Mhz *\n") == 2400.0
    assert kd.current_mhz("0: 500Mhz\n1: 2400Mhz\n") is None
