"""Launch kernels of the workloads a few times each, for hardware-counter runs.

    python3 paper_2606_09200_amd/kernel_driver.py --workload cb --kernel gemm --launches 5
    python3 paper_2606_09200_amd/kernel_driver.py --jobs cb:gemm,a2a:gemm,cb:comm --launches 3

Synchronises after every launch so that each dispatch is measured on its own,
prints one line per launch naming its job (the order of the dispatches in the
profiler's output), then (unless --no-copy) runs one plain device-to-device
copy of --copy-mib MiB whose bytes are known exactly: the counter values it
reads give the scale factor between the counters and true HBM bytes.

    python3 paper_2606_09200_amd/kernel_driver.py --jobs cb:gemm,cb:torch_mm --sustain 4 --power

--sustain S instead launches each job back to back (batches of 100 between
synchronisations) for about S seconds and prints the mean time per launch;
with --power it also samples the board's power sensor (the hwmon power1_input
file of the GPU, in microwatts) every 50 ms, idle first, and prints the
median and maximum per job next to the board's power cap.
"""
import argparse
import glob
import os
import sys
import threading
import time

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import torch  # noqa: E402

from paper_2606_09200_amd import binding as occ  # noqa: E402
from paper_2606_09200_amd import inputs  # noqa: E402
from paper_2606_09200_amd.workloads import WORKLOADS  # noqa: E402


def make_job(workload, kernel, b_layout, variant, pad_kib, dev):
    """A no-argument callable launching one kernel of the workload, plus the
    tensors it keeps alive."""
    w = WORKLOADS[workload]
    if kernel in ("gemm", "torch_mm"):
        A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_b=w.std_b, seed_b=w.seed_b, device=dev)
        C = torch.empty((w.M, w.N), device=dev, dtype=torch.bfloat16)
        B = Bt.t().contiguous() if b_layout == "kn" else Bt
        del Bt
        if kernel == "gemm" and b_layout == "kn":
            return lambda: occ.occ_gemm_ex(A, B, C, lds_bytes=pad_kib << 10, variant=variant)
        if kernel == "gemm":
            return lambda: occ.occ_gemm_bt_ex(A, B, C, lds_bytes=pad_kib << 10, variant=variant)
        if b_layout == "kn":
            return lambda: torch.mm(A, B, out=C)
        return lambda: torch.mm(A, B.t(), out=C)
    if w.comm == "reduce_own":
        own = torch.randn(w.length, device=dev).to(torch.bfloat16)
        ch = inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev)
        out = torch.empty(w.length, device=dev)
        return lambda: occ.share_reduce_own(own, ch, out)
    if w.comm == "reduce":
        ch = inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev)
        out = torch.empty(w.length, device=dev)
        return lambda: occ.share_reduce(ch, out)
    src = inputs.permute_payload(w.nchunks, w.chunk_bytes, seed=2, device=dev)
    dst = torch.empty_like(src)
    perm = inputs.chunk_permutation(w.nchunks, seed=3)
    return lambda: occ.share_permute(src, dst, perm, w.chunk_bytes)


def power_files():
    """(power1_input, power1_cap) of the first GPU's hwmon node, or None."""
    for d in sorted(glob.glob("/sys/class/drm/card*/device/hwmon/hwmon*")):
        pin, cap = os.path.join(d, "power1_input"), os.path.join(d, "power1_cap")
        if os.path.exists(pin):
            return pin, (cap if os.path.exists(cap) else None)
    return None


class PowerSampler:
    """Samples power1_input (microwatts) every 50 ms on a thread, labelled
    with the phase set by the caller."""

    def __init__(self, path):
        self.path, self.phase, self.samples = path, "idle", []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            try:
                with open(self.path) as f:
                    self.samples.append((self.phase, float(f.read()) / 1e6))
            except (OSError, ValueError):
                pass
            time.sleep(0.05)

    def start(self):
        self._t.start()

    def stop(self):
        self._stop.set()
        self._t.join()

    def summary(self, phase):
        xs = sorted(w for p, w in self.samples if p == phase)
        if not xs:
            return "no samples"
        return "median %.0f W, max %.0f W over %d samples" % (xs[len(xs) // 2], xs[-1], len(xs))


def sustain(run, seconds):
    """Launch `run` back to back for about `seconds`; returns (launches, elapsed)."""
    run()
    torch.cuda.synchronize()
    n, t0 = 0, time.time()
    while time.time() - t0 < seconds:
        for _ in range(100):
            run()
        torch.cuda.synchronize()
        n += 100
    return n, time.time() - t0


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="cb", choices=sorted(WORKLOADS))
    ap.add_argument("--kernel", default="gemm", choices=["gemm", "comm", "torch_mm"],
                    help="torch_mm: the same GEMM through torch.mm (hipBLASLt), for comparison")
    ap.add_argument("--jobs", default=None,
                    help="comma list of workload:kernel pairs run one after the other (instead of "
                         "--workload/--kernel)")
    ap.add_argument("--launches", type=int, default=5)
    ap.add_argument("--pad-kib", type=int, default=0)
    ap.add_argument("--variant", type=int, default=0)
    ap.add_argument("--b-layout", default="kn", choices=["kn", "nk"],
                    help="B stored K x N (occ_gemm) or N x K (occ_gemm_bt)")
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--no-copy", action="store_true")
    ap.add_argument("--sustain", type=float, default=0.0,
                    help="launch each job back to back for this many seconds (no per-launch sync, no copy)")
    ap.add_argument("--power", action="store_true", help="with --sustain: sample the board power sensor")
    a = ap.parse_args(argv)
    dev = "cuda:0"
    jobs = [tuple(j.split(":")) for j in a.jobs.split(",")] if a.jobs else [(a.workload, a.kernel)]
    for wl, k in jobs:
        if wl not in WORKLOADS or k not in ("gemm", "comm", "torch_mm"):
            raise SystemExit("unknown job %s:%s" % (wl, k))
    if a.sustain > 0:
        sampler = None
        if a.power:
            pf = power_files()
            if pf is None:
                raise SystemExit("no hwmon power1_input file for the GPU")
            if pf[1]:
                with open(pf[1]) as f:
                    print("power cap %.0f W (%s)" % (float(f.read()) / 1e6, pf[1]), flush=True)
            sampler = PowerSampler(pf[0])
            sampler.start()
            time.sleep(2.0)
            print("idle: %s" % sampler.summary("idle"), flush=True)
        for i, (wl, k) in enumerate(jobs):
            run = make_job(wl, k, a.b_layout, a.variant, a.pad_kib, dev)
            if sampler:
                sampler.phase = i
            n, e = sustain(run, a.sustain)
            if sampler:
                sampler.phase = "gap"
            line = "job %s:%s %d launches in %.2f s, %.4f ms per launch" % (wl, k, n, e, 1e3 * e / n)
            if sampler:
                line += "; board power %s" % sampler.summary(i)
            print(line, flush=True)
            del run
            torch.cuda.empty_cache()
            time.sleep(1.0)
        if sampler:
            sampler.stop()
        return 0
    for wl, k in jobs:
        run = make_job(wl, k, a.b_layout, a.variant, a.pad_kib, dev)
        torch.cuda.synchronize()
        for i in range(a.launches):
            run()
            torch.cuda.synchronize()
            print("job %s:%s launch %d done" % (wl, k, i), flush=True)
        del run
        torch.cuda.empty_cache()
    if not a.no_copy:
        x = torch.ones(a.copy_mib << 18, device=dev)   # float32: MiB * 2^18 elements
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        print("copy of %d MiB done (%d bytes read, %d written)" % (a.copy_mib, a.copy_mib << 20, a.copy_mib << 20), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
