"""Launch kernels of the workloads a few times each, for hardware-counter runs.

    python3 paper_2606_09200_amd/kernel_driver.py --workload cb --kernel gemm --launches 5
    python3 paper_2606_09200_amd/kernel_driver.py --jobs cb:gemm,a2a:gemm,cb:comm --launches 3

Synchronises after every launch so that each dispatch is measured on its own,
prints one line per launch naming its job (the order of the dispatches in the
profiler's output), then (unless --no-copy) runs one plain device-to-device
copy of --copy-mib MiB whose bytes are known exactly: the counter values it
reads give the scale factor between the counters and true HBM bytes.
"""
import argparse
import os
import sys

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
    a = ap.parse_args(argv)
    dev = "cuda:0"
    jobs = [tuple(j.split(":")) for j in a.jobs.split(",")] if a.jobs else [(a.workload, a.kernel)]
    for wl, k in jobs:
        if wl not in WORKLOADS or k not in ("gemm", "comm", "torch_mm"):
            raise SystemExit("unknown job %s:%s" % (wl, k))
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
