"""Benchmark: sequential vs overlapped makespan of GEMM -> collective iterations.

One step is one pass of the whole hot path over one batch of synthetic input:
the sequential schedule (one stream, G0 C0 ... G9 C9), the overlapped schedule
(two streams, event per iteration, comm kernel at raised wave priority), and
an isolated pass timing each kernel -- n_iter = 10 iterations each, on the
compute-bound workload (GEMM 8192^3 bf16 with an 8 x 2^25 fp32 allreduce
share) unless --workload says otherwise.

Prints ONE JSON line on stdout.  Everything else goes to stderr.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "overlapped vs sequential makespan (ms, % reduction); GEMM MFMA %, reduce HBM %"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest(names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2606_09200_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if the
    kernel source is unchanged since they were taken; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
        e = t[kernel][workload]
        if e["source_digest"] != source_digest(e["sources"]):
            return None
        return e["hbm_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


def make_inputs(w, dev):
    import torch
    from paper_2606_09200_amd import inputs
    A, B = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_a=w.std_a, std_b=w.std_b,
                                seed_b=w.seed_b, device=dev)
    if w.comm == "reduce_own":
        # one GEMM output per iteration; each iteration's collective reduces its own
        C = torch.empty((w.n_iter, w.M, w.N), device=dev, dtype=torch.bfloat16)
        comm = dict(bufs=inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev),
                    out=torch.empty(w.length, device=dev), reduce_own=True)
        return A, B, C, comm
    C = torch.empty((w.M, w.N), device=dev, dtype=torch.bfloat16)
    if w.comm == "reduce":
        comm = dict(bufs=inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=dev),
                    out=torch.empty(w.length, device=dev))
    else:
        src = inputs.permute_payload(w.nchunks, w.chunk_bytes, seed=2, device=dev)
        comm = dict(src=src, dst=torch.empty_like(src),
                    perm=inputs.chunk_permutation(w.nchunks, seed=3), chunk_bytes=w.chunk_bytes)
    return A, B, C, comm


def cpu_baseline(w, A, B, C, comm, budget_s, b_layout="nk"):
    """The oracle, as it stands, on a bounded sample of the same step, scaled
    to one sequential pass of n_iter iterations (ms)."""
    import numpy as np
    import torch
    import oracle
    Ah = A.view(torch.int16).cpu().numpy().view(np.uint16)
    Bh = B.view(torch.int16).cpu().numpy().view(np.uint16)
    cores = oracle.num_threads()   # the threads the oracle's loops actually run on
    # GEMM: whole-K 64x64 output tiles until about half the budget is spent
    t0 = time.perf_counter()
    tiles = 0
    rng = np.random.default_rng(0)
    while time.perf_counter() - t0 < budget_s / 2 and tiles < 4096:
        m0 = int(rng.integers(0, max(1, w.M - 64 + 1))) if w.M > 64 else 0
        n0 = int(rng.integers(0, max(1, w.N - 64 + 1))) if w.N > 64 else 0
        oracle.gemm_bf16(Ah, Bh, w.M, w.N, w.K, b_layout=b_layout, rows=(m0, min(w.M, m0 + 64)),
                         cols=(n0, min(w.N, n0 + 64)))
        tiles += 1
    t_gemm_sample = time.perf_counter() - t0
    macs_sample = tiles * min(64, w.M) * min(64, w.N) * w.K
    gemm_full_s = t_gemm_sample * (w.M * w.N * w.K) / macs_sample
    # comm: a contiguous slice of the same payload
    if w.comm == "reduce_own":
        n = min(w.length, 1 << 22)
        own = C[0].reshape(-1)[:n].cpu()
        sl = comm["bufs"][:, :n].cpu().numpy()
        t1 = time.perf_counter()
        oracle.chunk_sum_own_f32(own, sl)
        comm_full_s = (time.perf_counter() - t1) * w.length / n
        comm_desc = "bf16 own term + %d x %d fp32 chunk sum" % (w.nchunks, n)
    elif w.comm == "reduce":
        ch = comm["bufs"]
        n = min(w.length, 1 << 22)
        sl = ch[:, :n].cpu().numpy()
        t1 = time.perf_counter()
        oracle.chunk_sum_f32(sl)
        comm_full_s = (time.perf_counter() - t1) * w.length / n
        comm_desc = "%d x %d fp32 chunk sum" % (w.nchunks, n)
    else:
        src = comm["src"].cpu().numpy()
        t1 = time.perf_counter()
        oracle.permute_chunks(src, comm["perm"].numpy(), w.chunk_bytes)
        comm_full_s = time.perf_counter() - t1
        comm_desc = "full %d x %d B permutation" % (w.nchunks, w.chunk_bytes)
    step_ms = 1e3 * w.n_iter * (gemm_full_s + comm_full_s)
    return {
        "value": round(step_ms, 3),
        "unit": "ms (sequential makespan of %d GEMM->collective iterations, extrapolated)" % w.n_iter,
        "cores": cores,
        "kind": "oracle",
        "sample": "%d whole-K 64x64 GEMM output tiles (%.2f s) + %s, scaled per MAC / per element"
                  % (tiles, t_gemm_sample, comm_desc),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="cb", choices=["tiny", "cb", "mb", "a2a", "cb_own"])
    ap.add_argument("--pad-kib", type=int, default=0, help="extra LDS per GEMM workgroup")
    ap.add_argument("--priority", type=int, default=3, help="comm kernel wave priority 0..3")
    ap.add_argument("--variant", type=int, default=0, help="GEMM kernel variant (0 = auto)")
    ap.add_argument("--gemm-grid", type=int, default=0, help="persistent GEMM grid cap (0 = off)")
    ap.add_argument("--comm-wgs", type=int, default=0)
    ap.add_argument("--b-layout", default="nk", choices=["nk", "kn"],
                    help="GEMM B stored N x K (C = A B^T, occ_gemm) or K x N (C = A B, occ_gemm_kn)")
    ap.add_argument("--comm-rate-gbs", type=float, default=0.0,
                    help="bandwidth pacing of the collective in the overlapped schedule (0 = off)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the overlap method is per device and the library "
              "has no multi-GPU path; run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_09200_amd import binding as occ
    from paper_2606_09200_amd.workloads import WORKLOADS

    w = WORKLOADS[args.workload]
    dev = "cuda:0"
    torch.cuda.set_device(0)
    A, B, C, comm = make_inputs(w, dev)
    if args.b_layout == "kn":
        B = B.t().contiguous()  # the same matrix op(B), stored K x N
    torch.cuda.synchronize()
    knobs = dict(lds_bytes=args.pad_kib << 10, gemm_variant=args.variant, gemm_grid=args.gemm_grid,
                 comm_wgs=args.comm_wgs, comm_priority=args.priority, n_iter=w.n_iter,
                 comm_rate_gbs=args.comm_rate_gbs, b_layout=args.b_layout)

    # untimed warmup steps, then exactly `steps` timed steps
    occ.run_overlap(A, B, C, reps=args.warmup, warmup=0, **knobs, **comm) if args.warmup > 0 else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = occ.run_overlap(A, B, C, reps=args.steps, warmup=0, **knobs, **comm)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # the same overlapped schedule at normal comm priority (the paper's
    # baseline overlap) for the Norm. time of Section 4.2 / Fig. 3
    knobs_lo = dict(knobs, comm_priority=0)
    r_lo = occ.run_overlap(A, B, C, reps=max(3, args.steps // 2), warmup=1, flags=occ.OCC_RUN_OVL,
                           **knobs_lo, **comm)
    torch.cuda.synchronize()

    # kernel timeline and per-workgroup trace of one more overlapped pass:
    # overlap rate (Section 4.2), co-residency, and the GEMM workgroups'
    # lifetime and engine clock with and without the collective running
    from paper_2606_09200_amd import trace
    tl = torch.zeros(4 * w.n_iter, dtype=torch.int64, device=dev)
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * 40 * 1024, dtype=torch.int32, device=dev)
    occ.run_overlap(A, B, C, reps=1, warmup=0, flags=occ.OCC_RUN_OVL, timeline=tl, wg_trace=wt,
                    **knobs, **comm)
    torch.cuda.synchronize()
    g_iv, c_iv = trace.intervals(tl.cpu(), w.n_iter)
    overlap_rate = trace.overlap_rate(g_iv, c_iv)
    recs = occ.decode_wg_trace(wt)
    inter = trace.interference(recs, c_iv)
    cores = trace.coresidency(recs)
    resid = trace.residency(recs)

    # the same GEMM through torch.mm (hipBLASLt) on the same operands: a
    # same-run reference for the GEMM, context only
    C2 = C[0] if C.dim() == 3 else C
    ref_mm = (lambda: torch.mm(A, B.t(), out=C2)) if args.b_layout == "nk" else (lambda: torch.mm(A, B, out=C2))
    for _ in range(3):
        ref_mm()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        ref_mm()
    e1.record()
    torch.cuda.synchronize()
    hipblaslt_ms = e0.elapsed_time(e1) / 10

    # a plain 1 GiB device-to-device copy: a measured HBM ceiling beside the spec peak
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * src.numel() * 4 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst

    # Link-bound emulation (OCC_RUN_PACE_ALL): the local collective paced in
    # both schedules so that it lasts as long as one GEMM, as a collective
    # bound by inter-GPU links would on a multi-GPU node.  Reported beside
    # the headline number, never as it.
    emu_rate = max(occ.MIN_COMM_RATE_GBS, w.comm_bytes / (r["t_gemm_ms"] * 1e-3) / 1e9)
    emu = {}
    for prio in sorted({args.priority, 0}):
        e = occ.run_overlap(A, B, C, reps=max(3, args.steps // 2), warmup=1,
                            flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL | occ.OCC_RUN_PACE_ALL,
                            **dict(knobs, comm_priority=prio, comm_rate_gbs=emu_rate), **comm)
        emu[prio] = e
    torch.cuda.synchronize()

    gemm_tflops = w.gemm_flops / (r["t_gemm_ms"] * 1e-3) / 1e12
    comm_gbs = w.comm_bytes / (r["t_comm_ms"] * 1e-3) / 1e9
    plan = occ.occ_gemm_plan_query(w.M, w.N, w.K, args.pad_kib << 10, args.variant, args.gemm_grid,
                                   b_layout=args.b_layout)
    gemm_name = "occ_gemm" if args.b_layout == "nk" else "occ_gemm_kn"
    traffic_key = w.name if args.b_layout == "nk" else w.name + "_kn"
    gemm_bound_mb = w.M <= 16
    dominant_gemm = r["t_gemm_ms"] >= r["t_comm_ms"]
    if dominant_gemm and not gemm_bound_mb:
        roof = {"bound": "mfma", "achieved": round(gemm_tflops, 1), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(gemm_tflops / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic("gemm", traffic_key), "kernel": "%s variant %d" % (gemm_name, plan["kernel_id"])}
    elif dominant_gemm:
        gbs = w.gemm_bytes / (r["t_gemm_ms"] * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic("gemm", traffic_key),
                "kernel": "%s variant %d" % (gemm_name, plan["kernel_id"])}
    else:
        roof = {"bound": "hbm", "achieved": round(comm_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(comm_gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic("comm", w.name),
                "kernel": "share_" + w.comm}

    line = {
        "metric": METRIC,
        "value": round(r["reduction_pct"], 3),
        "unit": "% makespan reduction, overlapped vs sequential (100*(1-TimeRatio))",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * wall / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 (fp32 accumulate) + f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: bf16 GEMM %dx%dx%d (B as %s) + %s, %d iterations per schedule"
                        % (w.name, w.M, w.N, w.K, "N x K" if args.b_layout == "nk" else "K x N",
                           ("share_reduce %d x %d fp32" % (w.nchunks, w.length)) if w.comm == "reduce"
                           else ("share_reduce_own of C_i + %d x %d fp32" % (w.nchunks, w.length))
                           if w.comm == "reduce_own"
                           else ("share_permute %d x %d B" % (w.nchunks, w.chunk_bytes)), w.n_iter),
            "lds_pad_bytes": args.pad_kib << 10,
            "comm_wave_priority": args.priority,
            "gemm_variant": plan["kernel_id"],
            "gemm_tile": "%dx%dx%d" % (plan["tile_m"], plan["tile_n"], plan["tile_k"]),
            "gemm_tile_lds_bytes": plan["tile_lds_bytes"],
            "gemm_wg_per_cu": plan["wg_per_cu"],
            "gemm_grid": plan["grid"],
            "comm_wgs": r["comm_wgs"],
            "comm_rate_gbs": args.comm_rate_gbs,
            "parallelism": "single GPU",
        },
        "t_seq_ms": round(r["t_seq_ms"], 4),
        "t_ovl_ms": round(r["t_ovl_ms"], 4),
        "t_seq_median_ms": round(r["t_seq_median_ms"], 4),
        "t_ovl_median_ms": round(r["t_ovl_median_ms"], 4),
        "t_seq_std_ms": round(r["t_seq_std_ms"], 4),
        "t_ovl_std_ms": round(r["t_ovl_std_ms"], 4),
        "time_ratio": round(r["t_ovl_ms"] / r["t_seq_ms"], 4),
        "t_gemm_ms": round(r["t_gemm_ms"], 4),
        "t_comm_ms": round(r["t_comm_ms"], 4),
        "ideal_ovl_ms": round(w.n_iter * max(r["t_gemm_ms"], r["t_comm_ms"]) + min(r["t_gemm_ms"], r["t_comm_ms"]), 4),
        "gemm_tflops": round(gemm_tflops, 1),
        "gemm_hipblaslt_tflops": round(w.gemm_flops / (hipblaslt_ms * 1e-3) / 1e12, 1),
        "gemm_mfma_frac": round(gemm_tflops / PEAK_BF16_TFLOPS, 4),
        "comm_gbs": round(comm_gbs, 1),
        "comm_hbm_frac": round(comm_gbs / PEAK_HBM_GBS, 4),
        "hbm_copy_gbs": round(copy_gbs, 1),
        "comm_copy_frac": round(comm_gbs / copy_gbs, 4),
        "overlap_rate": round(overlap_rate, 4),
        "comm_coresident": None if cores is None else round(cores, 4),
        "gemm_wg_per_cu_achieved": resid,
        "gemm_wg": inter,
        "t_ovl_normal_priority_ms": round(r_lo["t_ovl_ms"], 4),
        "reduction_pct_normal_priority": round(100.0 * (1.0 - r_lo["t_ovl_ms"] / r["t_seq_ms"]), 3),
        "norm_time_priority": round(r["t_ovl_ms"] / r_lo["t_ovl_ms"], 4),
        "link_bound_emulation": {
            "comm_rate_gbs": round(emu_rate, 1),
            "t_seq_ms": round(emu[args.priority]["t_seq_ms"], 4),
            "t_ovl_ms": round(emu[args.priority]["t_ovl_ms"], 4),
            "reduction_pct": round(emu[args.priority]["reduction_pct"], 3),
            "t_ovl_normal_priority_ms": round(emu[0]["t_ovl_ms"], 4),
            "reduction_pct_normal_priority": round(100.0 * (1.0 - emu[0]["t_ovl_ms"] / emu[args.priority]["t_seq_ms"]), 3),
            "note": "collective paced in both schedules to last one GEMM (OCC_RUN_PACE_ALL); not the headline value",
        },
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        log("cpu baseline: timing the oracle on a bounded sample ...")
        line["cpu_baseline"] = cpu_baseline(w, A, B, C, comm, args.cpu_budget, args.b_layout)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
