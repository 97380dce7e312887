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
synchronisations; one call for the seq / ovl schedule jobs) for about S
seconds and prints the mean time per launch; with --power it also samples the
board's power sensor (the hwmon power1_input file of the GPU, in microwatts)
and the current engine clock (the starred line of pp_dpm_sclk) every 50 ms,
idle first, and prints their medians and the maximum power per job next to
the board's power cap.
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
    tensors it keeps alive.  kernel "seq" / "ovl": one run_overlap call of the
    workload's sequential / overlapped schedule (n_iter iterations, 3 timed
    passes, comm wave priority 0)."""
    w = WORKLOADS[workload]
    if kernel in ("seq", "ovl"):
        if w.comm == "reduce_own":
            raise SystemExit("seq/ovl jobs: reduce and permute workloads only")
        A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_b=w.std_b, seed_b=w.seed_b, device=dev)
        B = Bt.t().contiguous() if b_layout == "kn" else Bt
        del Bt
        C = torch.empty((w.M, w.N), device=dev, dtype=torch.bfloat16)
        if w.comm == "reduce":
            comm = dict(bufs=inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev),
                        out=torch.empty(w.length, device=dev))
        else:
            src = inputs.permute_payload(w.nchunks, w.chunk_bytes, seed=2, device=dev)
            comm = dict(src=src, dst=torch.empty_like(src), perm=inputs.chunk_permutation(w.nchunks, seed=3),
                        chunk_bytes=w.chunk_bytes)
        flags = occ.OCC_RUN_SEQ if kernel == "seq" else occ.OCC_RUN_OVL
        return lambda: occ.run_overlap(A, B, C, n_iter=w.n_iter, reps=3, warmup=0, flags=flags, comm_priority=0,
                                       lds_bytes=pad_kib << 10, gemm_variant=variant, b_layout=b_layout, **comm)
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
    """(power1_input, power1_cap, pp_dpm_sclk) of the first GPU with a hwmon
    power sensor (the last two None where absent), or None."""
    for d in sorted(glob.glob("/sys/class/drm/card*/device/hwmon/hwmon*")):
        pin, cap = os.path.join(d, "power1_input"), os.path.join(d, "power1_cap")
        sclk = os.path.join(os.path.dirname(os.path.dirname(d)), "pp_dpm_sclk")
        if os.path.exists(pin):
            return pin, (cap if os.path.exists(cap) else None), (sclk if os.path.exists(sclk) else None)
    return None


def current_mhz(text):
    """The starred (current) level of a pp_dpm_sclk listing, in MHz, or None."""
    for line in text.splitlines():
        if line.rstrip().endswith("*"):
            f = line.split(":", 1)[-1].strip().rstrip("*").strip().lower().replace("mhz", "")
            try:
                return float(f)
            except ValueError:
                return None
    return None


class PowerSampler:
    """Samples power1_input (microwatts) and, if given, the current engine
    clock from pp_dpm_sclk every 50 ms on a thread, labelled with the phase
    set by the caller."""

    def __init__(self, path, sclk_path=None):
        self.path, self.sclk_path, self.phase, self.samples, self.clocks = path, sclk_path, "idle", [], []
        self._stop = threading.Event()
        self._t = threading.Thread(target=self._run, daemon=True)

    def _run(self):
        while not self._stop.is_set():
            try:
                with open(self.path) as f:
                    self.samples.append((self.phase, float(f.read()) / 1e6))
            except (OSError, ValueError):
                pass
            if self.sclk_path:
                try:
                    with open(self.sclk_path) as f:
                        mhz = current_mhz(f.read())
                    if mhz is not None:
                        self.clocks.append((self.phase, mhz))
                except OSError:
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
        line = "median %.0f W, max %.0f W over %d samples" % (xs[len(xs) // 2], xs[-1], len(xs))
        cs = sorted(c for p, c in self.clocks if p == phase)
        if cs:
            line += "; engine clock median %.0f MHz" % cs[len(cs) // 2]
        return line


def sustain(run, seconds, batch=100):
    """Launch `run` back to back for about `seconds`, `batch` calls between
    synchronisations; returns (launches, elapsed)."""
    run()
    torch.cuda.synchronize()
    n, t0 = 0, time.time()
    while time.time() - t0 < seconds:
        for _ in range(batch):
            run()
        torch.cuda.synchronize()
        n += batch
    return n, time.time() - t0


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="cb", choices=sorted(WORKLOADS))
    ap.add_argument("--kernel", default="gemm", choices=["gemm", "comm", "torch_mm", "seq", "ovl"],
                    help="torch_mm: the same GEMM through torch.mm (hipBLASLt), for comparison; seq / ovl: "
                         "one run_overlap call of the sequential / overlapped schedule")
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
        if wl not in WORKLOADS or k not in ("gemm", "comm", "torch_mm", "seq", "ovl"):
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
            sampler = PowerSampler(pf[0], pf[2])
            sampler.start()
            time.sleep(2.0)
            print("idle: %s" % sampler.summary("idle"), flush=True)
        for i, (wl, k) in enumerate(jobs):
            run = make_job(wl, k, a.b_layout, a.variant, a.pad_kib, dev)
            if sampler:
                sampler.phase = i
            n, e = sustain(run, a.sustain, 1 if k in ("seq", "ovl") else 100)
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
