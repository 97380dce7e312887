"""Launch one kernel of a workload a few times, for hardware-counter runs.

    python3 paper_2606_09200_amd/kernel_driver.py --workload cb --kernel gemm --launches 5

Synchronises after every launch so that each dispatch is measured on its own,
then (unless --no-copy) runs one plain device-to-device copy of --copy-mib MiB
whose bytes are known exactly: the counter values it reads give the scale
factor between the counters and true HBM bytes.
"""
import argparse
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import torch  # noqa: E402

from paper_2606_09200_amd import binding as occ  # noqa: E402
from paper_2606_09200_amd import inputs  # noqa: E402
from paper_2606_09200_amd.workloads import WORKLOADS  # noqa: E402


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="cb", choices=sorted(WORKLOADS))
    ap.add_argument("--kernel", default="gemm", choices=["gemm", "comm", "torch_mm"],
                    help="torch_mm: the same GEMM through torch.mm (hipBLASLt), for comparison")
    ap.add_argument("--launches", type=int, default=5)
    ap.add_argument("--pad-kib", type=int, default=0)
    ap.add_argument("--variant", type=int, default=0)
    ap.add_argument("--b-layout", default="kn", choices=["kn", "nk"],
                    help="B stored K x N (occ_gemm) or N x K (occ_gemm_bt)")
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--no-copy", action="store_true")
    a = ap.parse_args(argv)
    w = WORKLOADS[a.workload]
    dev = "cuda:0"
    if a.kernel in ("gemm", "torch_mm"):
        A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_b=w.std_b, seed_b=w.seed_b, device=dev)
        C = torch.empty((w.M, w.N), device=dev, dtype=torch.bfloat16)
        B = Bt.t().contiguous() if a.b_layout == "kn" else Bt
        del Bt
        if a.kernel == "gemm" and a.b_layout == "kn":
            run = lambda: occ.occ_gemm_ex(A, B, C, lds_bytes=a.pad_kib << 10, variant=a.variant)
        elif a.kernel == "gemm":
            run = lambda: occ.occ_gemm_bt_ex(A, B, C, lds_bytes=a.pad_kib << 10, variant=a.variant)
        elif a.b_layout == "kn":
            run = lambda: torch.mm(A, B, out=C)
        else:
            run = lambda: torch.mm(A, B.t(), out=C)
    elif w.comm == "reduce_own":
        own = torch.randn(w.length, device=dev).to(torch.bfloat16)
        ch = inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev)
        out = torch.empty(w.length, device=dev)
        run = lambda: occ.share_reduce_own(own, ch, out)
    elif w.comm == "reduce":
        ch = inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev)
        out = torch.empty(w.length, device=dev)
        run = lambda: occ.share_reduce(ch, out)
    else:
        src = inputs.permute_payload(w.nchunks, w.chunk_bytes, seed=2, device=dev)
        dst = torch.empty_like(src)
        perm = inputs.chunk_permutation(w.nchunks, seed=3)
        run = lambda: occ.share_permute(src, dst, perm, w.chunk_bytes)
    torch.cuda.synchronize()
    for i in range(a.launches):
        run()
        torch.cuda.synchronize()
        print("launch %d done" % i, flush=True)
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
