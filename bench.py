"""Benchmark: sequential vs overlapped makespan of GEMM -> collective iterations.

One step is one pass of the whole hot path over one batch of synthetic input:
the sequential schedule (one stream, G0 C0 ... G9 C9), the overlapped schedule
(two streams, a dependency per iteration, comm kernel at raised wave
priority), and an isolated pass timing each kernel -- n_iter = 10 iterations
each.  The headline is the compute-bound workload (GEMM 8192^3 bf16 through
occ_gemm, B stored K x N, with an 8 x 2^25 fp32 allreduce share) unless
--workload says otherwise; the same line carries every workload of the
evaluation under "configs": tiny, cb, mb, a2a and the pad x priority sweep,
each with its makespans, its dominant kernel's roofline and the CPU oracle
timed on a bounded sample of it.

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
CONFIGS = ("tiny", "cb", "mb", "a2a", "sweep")
# Knobs of the workloads beyond the defaults.  The tiny pair's kernels are
# shorter than the host's issue time for an event, so it runs with the
# device counter dependency and a lightweight, low-occupancy collective (one
# workgroup per four CUs); its record also carries the default comm grid.
CONFIG_DEP = {"tiny": "counter"}
CONFIG_COMM_WGS_PER_CU = {"tiny": 0.25}
# Extra GEMM LDS pads a workload's record also reports, at both comm
# priorities (the tiny pair's definition: pad {0, 64 KiB} x priority).
CONFIG_EXTRA_PADS_KIB = {"tiny": (64,)}
# GEMM tile of a workload's record where it is not the library's automatic
# choice: the tiny pair runs the paper's opt2 tile (Table 1, 16 KiB, so the
# 64 KiB pad leaves two workgroups per CU); its record also reports the
# sequential schedule with the automatic choice.
CONFIG_GEMM_VARIANT = {"tiny": {"kn": 37, "nk": 7}}
SWEEP_PADS_KIB = (0, 16, 32, 64, 96, 128)
SWEEP_TILES = ((0, "default tile"), (37, "opt2 64x64x64"))


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


def make_inputs(w, dev, b_layout="kn"):
    import torch
    from paper_2606_09200_amd import inputs
    A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_a=w.std_a, std_b=w.std_b,
                                 seed_b=w.seed_b, device=dev)
    B = Bt.t().contiguous() if b_layout == "kn" else Bt   # the same op(B) in the chosen layout
    del Bt
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


def describe(w, b_layout):
    comm = (("share_reduce %d x %d fp32" % (w.nchunks, w.length)) if w.comm == "reduce"
            else ("share_reduce_own of C_i + %d x %d fp32" % (w.nchunks, w.length)) if w.comm == "reduce_own"
            else ("share_permute %d x %d B" % (w.nchunks, w.chunk_bytes)))
    return "%s: bf16 GEMM %dx%dx%d (%s) + %s, %d iterations per schedule" % (
        w.name, w.M, w.N, w.K, "occ_gemm, B K x N" if b_layout == "kn" else "occ_gemm_bt, B N x K",
        comm, w.n_iter)


def cpu_baseline(w, A, B, C, comm, budget_s, b_layout="kn"):
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


def roofline(w, r, kernel_name, b_layout):
    """The dominant kernel's achieved rate against its bound: algorithmic work
    per launch over the mean launch time of the isolated pass (HIP events on
    the stream the kernels run on)."""
    gemm_dominant = r["t_gemm_ms"] >= r["t_comm_ms"]
    traffic_kernel = "gemm" if b_layout == "kn" else "gemm_bt"
    if gemm_dominant and w.M > 16:
        tf = w.gemm_flops / (r["t_gemm_ms"] * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": round(tf, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(traffic_kernel, w.name),
                "kernel": kernel_name, "work_per_launch": "%.4g flop" % w.gemm_flops}
    if gemm_dominant:
        gbs = w.gemm_bytes / (r["t_gemm_ms"] * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic(traffic_kernel, w.name),
                "kernel": kernel_name, "work_per_launch": "%.4g B" % w.gemm_bytes}
    gbs = w.comm_bytes / (r["t_comm_ms"] * 1e-3) / 1e9
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": measured_traffic("comm", w.name),
            "kernel": "share_" + w.comm, "work_per_launch": "%.4g B" % w.comm_bytes}


def measure_workload(occ, w, A, B, C, comm, knobs, steps, warmup, dep):
    """Makespans at the configured comm priority and at normal priority, the
    other dependency kind, the overlap rate and workgroup statistics of one
    traced overlapped pass."""
    import torch
    from paper_2606_09200_amd import trace
    dev = "cuda:0"
    knobs = dict(knobs, dep=dep)
    r = occ.run_overlap(A, B, C, reps=steps, warmup=warmup, **knobs, **comm)
    torch.cuda.synchronize()
    lo_reps = max(3, steps // 2)
    r_lo = occ.run_overlap(A, B, C, reps=lo_reps, warmup=1, flags=occ.OCC_RUN_OVL,
                           **dict(knobs, comm_priority=0), **comm)
    other = "event" if dep == "counter" else "counter"
    try:
        r_alt = occ.run_overlap(A, B, C, reps=lo_reps, warmup=1, flags=occ.OCC_RUN_OVL,
                                **dict(knobs, dep=other), **comm)
    except occ.OccError as e:       # e.g. more comm workgroups than the counter allows
        r_alt = {"error": str(e)}
    tl = torch.zeros(4 * w.n_iter, dtype=torch.int64, device=dev)
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * 40 * 1024, dtype=torch.int32, device=dev)
    occ.run_overlap(A, B, C, reps=1, warmup=0, flags=occ.OCC_RUN_OVL, timeline=tl, wg_trace=wt,
                    **knobs, **comm)
    torch.cuda.synchronize()
    g_iv, c_iv = trace.intervals(tl.cpu(), w.n_iter)
    recs = occ.decode_wg_trace(wt)
    rec = {
        "dep": dep,
        "t_seq_ms": round(r["t_seq_ms"], 4),
        "t_ovl_ms": round(r["t_ovl_ms"], 4),
        "reduction_pct": round(r["reduction_pct"], 3),
        "t_seq_median_ms": round(r["t_seq_median_ms"], 4),
        "t_ovl_median_ms": round(r["t_ovl_median_ms"], 4),
        "t_seq_std_ms": round(r["t_seq_std_ms"], 4),
        "t_ovl_std_ms": round(r["t_ovl_std_ms"], 4),
        "time_ratio": round(r["t_ovl_ms"] / r["t_seq_ms"], 4),
        "t_gemm_ms": round(r["t_gemm_ms"], 4),
        "t_comm_ms": round(r["t_comm_ms"], 4),
        "ideal_ovl_ms": round(w.n_iter * max(r["t_gemm_ms"], r["t_comm_ms"]) + min(r["t_gemm_ms"], r["t_comm_ms"]), 4),
        "t_ovl_normal_priority_ms": round(r_lo["t_ovl_ms"], 4),
        "reduction_pct_normal_priority": round(100.0 * (1.0 - r_lo["t_ovl_ms"] / r["t_seq_ms"]), 3),
        "norm_time_priority": round(r["t_ovl_ms"] / r_lo["t_ovl_ms"], 4),
        "t_ovl_%s_dep_ms" % other: (round(r_alt["t_ovl_ms"], 4) if "t_ovl_ms" in r_alt else r_alt["error"]),
        "overlap_rate": round(trace.overlap_rate(g_iv, c_iv), 4),
        "comm_coresident": trace.coresidency(recs),
        "gemm_wg_per_cu_achieved": trace.residency(recs),
        "gemm_wg": trace.interference(recs, c_iv),
        "comm_wgs": r["comm_wgs"],
        "gemm_wg_per_cu": r["gemm_wg_per_cu"],
        "gemm_tflops": round(w.gemm_flops / (r["t_gemm_ms"] * 1e-3) / 1e12, 1),
        "gemm_mfma_frac": round(w.gemm_flops / (r["t_gemm_ms"] * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "gemm_hbm_frac": round(w.gemm_bytes / (r["t_gemm_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
        "comm_gbs": round(w.comm_bytes / (r["t_comm_ms"] * 1e-3) / 1e9, 1),
        "comm_hbm_frac": round(w.comm_bytes / (r["t_comm_ms"] * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
    }
    if rec["comm_coresident"] is not None:
        rec["comm_coresident"] = round(rec["comm_coresident"], 4)
    return r, rec


def tuned(occ, w, A, B, C, comm, steps, b_layout="kn"):
    """occ_overlap_tune's choice for the workload and the makespans it gives."""
    knobs, r, prefer_seq = occ.occ_overlap_tune(A, B, C, n_iter=w.n_iter, reps=max(3, steps // 2), warmup=2,
                                                tune_reps=3, b_layout=b_layout, **comm)
    return {"knobs": knobs, "t_seq_ms": round(r["t_seq_median_ms"], 4), "t_ovl_ms": round(r["t_ovl_median_ms"], 4),
            "reduction_pct": round(100.0 * (1.0 - r["t_ovl_median_ms"] / r["t_seq_median_ms"]), 3),
            "prefer_sequential": prefer_seq, "note": "medians of the tuned setting's own run"}


def sweep_points(occ, w, A, B, C, comm, b_layout):
    """Config 5: the cb pair over the extra LDS pad x comm wave priority, with
    the default tile (only small pads fit beside its 128 KiB) and the paper's
    opt2 tile (whose residency the pad sets over the whole range)."""
    import torch
    rows = []
    for variant, tile in SWEEP_TILES:
        for pad_kib in SWEEP_PADS_KIB:
            plan = occ.occ_gemm_plan_query(w.M, w.N, w.K, pad_kib << 10, variant, b_layout=b_layout)
            for prio in (0, 3):
                row = {"tile": tile, "gemm_variant": plan["kernel_id"], "pad_kib": pad_kib, "comm_priority": prio,
                       "gemm_tile_lds": plan["tile_lds_bytes"], "feasible": plan["feasible"],
                       "gemm_wg_per_cu": plan["wg_per_cu"] if plan["feasible"] else 0}
                if plan["feasible"]:
                    r = occ.run_overlap(A, B, C, reps=3, warmup=1, lds_bytes=pad_kib << 10, gemm_variant=variant,
                                        comm_priority=prio, n_iter=w.n_iter, b_layout=b_layout, **comm)
                    torch.cuda.synchronize()
                    tf = w.gemm_flops / (r["t_gemm_ms"] * 1e-3) / 1e12
                    row.update({"t_seq_ms": round(r["t_seq_ms"], 4), "t_ovl_ms": round(r["t_ovl_ms"], 4),
                                "reduction_pct": round(r["reduction_pct"], 3),
                                "t_gemm_ms": round(r["t_gemm_ms"], 4), "gemm_mfma_frac": round(tf / PEAK_BF16_TFLOPS, 4),
                                "comm_gbs": round(w.comm_bytes / (r["t_comm_ms"] * 1e-3) / 1e9, 1)})
                rows.append(row)
                log("sweep", json.dumps(row))
    for row in rows:                 # Norm. time: high over normal priority at the same point
        if row.get("comm_priority") == 3 and "t_ovl_ms" in row:
            base = [x for x in rows if x["tile"] == row["tile"] and x["pad_kib"] == row["pad_kib"]
                    and x["comm_priority"] == 0 and "t_ovl_ms" in x]
            if base:
                row["norm_time_priority"] = round(row["t_ovl_ms"] / base[0]["t_ovl_ms"], 4)
    feas = [x for x in rows if "t_ovl_ms" in x]
    best = min(feas, key=lambda x: x["t_ovl_ms"]) if feas else None
    return {"workload": describe(w, b_layout) + "; pad x comm priority, two tiles",
            "points": rows,
            "best": None if best is None else {k: best[k] for k in ("tile", "pad_kib", "comm_priority", "t_ovl_ms",
                                                                 "reduction_pct")},
            "reduction_pct_range": None if not feas else [min(x["reduction_pct"] for x in feas),
                                                         max(x["reduction_pct"] for x in feas)]}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="cb", choices=["tiny", "cb", "mb", "a2a", "cb_own"],
                    help="the headline workload")
    ap.add_argument("--configs", default=",".join(CONFIGS),
                    help="comma list of the workloads reported under 'configs' (or 'none')")
    ap.add_argument("--pad-kib", type=int, default=0, help="extra LDS per GEMM workgroup")
    ap.add_argument("--priority", type=int, default=3, help="comm kernel wave priority 0..3")
    ap.add_argument("--variant", type=int, default=0, help="GEMM kernel variant (0 = auto)")
    ap.add_argument("--gemm-grid", type=int, default=0, help="persistent GEMM grid cap (0 = off)")
    ap.add_argument("--comm-wgs", type=int, default=0)
    ap.add_argument("--b-layout", default="kn", choices=["kn", "nk"],
                    help="GEMM B stored K x N (C = A B, occ_gemm) or N x K (C = A B^T, occ_gemm_bt)")
    ap.add_argument("--dep", default=None, choices=["event", "counter"],
                    help="per-iteration dependency of the headline (default: the workload's own)")
    ap.add_argument("--comm-rate-gbs", type=float, default=0.0,
                    help="bandwidth pacing of the collective in the overlapped schedule (0 = off)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle work for the headline")
    ap.add_argument("--config-cpu-budget", type=float, default=3.0, help="seconds of oracle work per other config")
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
    A, B, C, comm = make_inputs(w, dev, args.b_layout)
    torch.cuda.synchronize()
    dep = args.dep or CONFIG_DEP.get(w.name, "event")
    # the workload's own knobs where the command line leaves them at 0
    variant = args.variant or CONFIG_GEMM_VARIANT.get(w.name, {}).get(args.b_layout, 0)
    num_cus = occ.occ_gemm_plan_query(w.M, w.N, w.K, 0, variant, b_layout=args.b_layout)["num_cus"]
    comm_wgs = args.comm_wgs or int(CONFIG_COMM_WGS_PER_CU.get(w.name, 0) * num_cus)
    knobs = dict(lds_bytes=args.pad_kib << 10, gemm_variant=variant, gemm_grid=args.gemm_grid,
                 comm_wgs=comm_wgs, comm_priority=args.priority, n_iter=w.n_iter,
                 comm_rate_gbs=args.comm_rate_gbs, b_layout=args.b_layout, dep=dep)
    gemm_name = "occ_gemm" if args.b_layout == "kn" else "occ_gemm_bt"

    # untimed warmup steps, then exactly `steps` timed steps
    log("headline %s: warm-up and %d timed steps" % (w.name, args.steps))
    if args.warmup > 0:
        occ.run_overlap(A, B, C, reps=args.warmup, warmup=0, **knobs, **comm)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    r = occ.run_overlap(A, B, C, reps=args.steps, warmup=0, **knobs, **comm)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    # the rest of the headline record (normal priority for the Norm. time of
    # Section 4.2 / Fig. 3, the other dependency, overlap rate, workgroups)
    _, rec = measure_workload(occ, w, A, B, C, comm, {k: v for k, v in knobs.items() if k != "dep"},
                              max(3, args.steps // 2), 2, dep)
    for k in ("t_seq_ms", "t_ovl_ms", "reduction_pct", "t_seq_median_ms", "t_ovl_median_ms", "t_seq_std_ms",
              "t_ovl_std_ms", "time_ratio", "t_gemm_ms", "t_comm_ms", "ideal_ovl_ms", "gemm_tflops",
              "gemm_mfma_frac", "gemm_hbm_frac", "comm_gbs", "comm_hbm_frac"):
        rec.pop(k, None)
    plan = occ.occ_gemm_plan_query(w.M, w.N, w.K, args.pad_kib << 10, variant, args.gemm_grid,
                                   b_layout=args.b_layout)

    # the same GEMM through torch.mm (hipBLASLt) on the same operands: a
    # same-run reference for the GEMM, context only.  Timed after half a
    # second of back-to-back calls: an idle chip needs tens of milliseconds
    # to reach its steady clock, and a short burst from idle reads 15-20 %
    # slow.
    C2 = C[0] if C.dim() == 3 else C
    ref_mm = (lambda: torch.mm(A, B, out=C2)) if args.b_layout == "kn" else (lambda: torch.mm(A, B.t(), out=C2))
    t_warm = time.time()
    while time.time() - t_warm < 0.5:
        for _ in range(20):
            ref_mm()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(20):
        ref_mm()
    e1.record()
    torch.cuda.synchronize()
    hipblaslt_ms = e0.elapsed_time(e1) / 20

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
        emu[prio] = occ.run_overlap(A, B, C, reps=max(3, args.steps // 2), warmup=1,
                                    flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL | occ.OCC_RUN_PACE_ALL,
                                    **dict(knobs, comm_priority=prio, comm_rate_gbs=emu_rate), **comm)
    torch.cuda.synchronize()

    gemm_tflops = w.gemm_flops / (r["t_gemm_ms"] * 1e-3) / 1e12
    comm_gbs = w.comm_bytes / (r["t_comm_ms"] * 1e-3) / 1e9
    kernel_name = "%s variant %d" % (gemm_name, plan["kernel_id"])
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
            "workload": describe(w, args.b_layout),
            "lds_pad_bytes": args.pad_kib << 10,
            "comm_wave_priority": args.priority,
            "dep": dep,
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
    }
    line.update(rec)
    line["link_bound_emulation"] = {
        "comm_rate_gbs": round(emu_rate, 1),
        "t_seq_ms": round(emu[args.priority]["t_seq_ms"], 4),
        "t_ovl_ms": round(emu[args.priority]["t_ovl_ms"], 4),
        "reduction_pct": round(emu[args.priority]["reduction_pct"], 3),
        "t_ovl_normal_priority_ms": round(emu[0]["t_ovl_ms"], 4),
        "reduction_pct_normal_priority": round(100.0 * (1.0 - emu[0]["t_ovl_ms"] / emu[args.priority]["t_seq_ms"]), 3),
        "note": "collective paced in both schedules to last one GEMM (OCC_RUN_PACE_ALL); not the headline value",
    }
    line["roofline"] = roofline(w, r, kernel_name, args.b_layout)
    if not args.no_cpu_baseline:
        log("cpu baseline: timing the oracle on a bounded sample ...")
        line["cpu_baseline"] = cpu_baseline(w, A, B, C, comm, args.cpu_budget, args.b_layout)
    log("tuner on the headline workload")
    line["tuned"] = tuned(occ, w, A, B, C, comm, args.steps, args.b_layout)
    headline = dict(line)

    # every workload of the evaluation, each with its own record
    configs = {}
    names = [] if args.configs == "none" else [c for c in args.configs.split(",") if c]
    del A, B, C, comm
    torch.cuda.empty_cache()
    for name in names:
        if name == "sweep":
            log("config sweep")
            ws = WORKLOADS["cb"]
            A, B, C, comm = make_inputs(ws, dev, args.b_layout)
            configs["sweep"] = sweep_points(occ, ws, A, B, C, comm, args.b_layout)
        elif name == w.name and args.b_layout == "kn":
            configs[name] = {k: headline[k] for k in headline if k not in (
                "metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "link_bound_emulation")}
            configs[name]["workload"] = headline["config"]["workload"]
            continue
        else:
            log("config %s" % name)
            wc = WORKLOADS[name]
            A, B, C, comm = make_inputs(wc, dev, "kn")
            torch.cuda.synchronize()
            cdep = CONFIG_DEP.get(name, "event")
            cvar = CONFIG_GEMM_VARIANT.get(name, {}).get("kn", 0)
            pc = occ.occ_gemm_plan_query(wc.M, wc.N, wc.K, 0, cvar)
            cwgs = int(CONFIG_COMM_WGS_PER_CU.get(name, 0) * pc["num_cus"])
            kn = dict(n_iter=wc.n_iter, comm_priority=3, b_layout="kn", comm_wgs=cwgs, gemm_variant=cvar)
            rc, rec = measure_workload(occ, wc, A, B, C, comm, kn, args.steps, args.warmup, cdep)
            rec = dict({"workload": describe(wc, "kn"), "gemm_variant": pc["kernel_id"]}, **rec)
            if cvar:
                # the sequential schedule with the library's automatic GEMM choice
                pa = occ.occ_gemm_plan_query(wc.M, wc.N, wc.K)
                ra = occ.run_overlap(A, B, C, reps=args.steps, warmup=args.warmup,
                                     flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_ISO, **dict(kn, gemm_variant=0, dep=cdep),
                                     **comm)
                rec["automatic_gemm_choice"] = {"gemm_variant": pa["kernel_id"],
                                                "t_seq_ms": round(ra["t_seq_median_ms"], 4),
                                                "t_gemm_ms": round(ra["t_gemm_ms"], 5), "note": "medians"}
            if cwgs:
                # the same pair with the library's default comm grid (one per CU)
                d = {}
                for dd in ("counter", "event"):
                    rd = occ.run_overlap(A, B, C, reps=args.steps, warmup=args.warmup, flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL,
                                         **dict(kn, comm_wgs=0, dep=dd), **comm)
                    d[dd] = {"t_seq_ms": round(rd["t_seq_median_ms"], 4), "t_ovl_ms": round(rd["t_ovl_median_ms"], 4),
                             "reduction_pct": round(100.0 * (1.0 - rd["t_ovl_median_ms"] / rd["t_seq_median_ms"]), 3)}
                rec["default_comm_grid"] = dict(d, comm_wgs=rd["comm_wgs"], note="medians")
            pads = []
            for pad_kib in CONFIG_EXTRA_PADS_KIB.get(name, ()):
                pp = occ.occ_gemm_plan_query(wc.M, wc.N, wc.K, pad_kib << 10, cvar)
                row = {"pad_kib": pad_kib, "gemm_wg_per_cu": pp["wg_per_cu"] if pp["feasible"] else 0}
                if pp["feasible"]:
                    rp = {}
                    for prio in (3, 0):
                        rp[prio] = occ.run_overlap(A, B, C, reps=args.steps, warmup=args.warmup,
                                                   flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL,
                                                   **dict(kn, lds_bytes=pad_kib << 10, comm_priority=prio, dep=cdep),
                                                   **comm)
                    row.update({"t_seq_ms": round(rp[3]["t_seq_median_ms"], 4),
                                "t_ovl_ms": round(rp[3]["t_ovl_median_ms"], 4),
                                "t_ovl_normal_priority_ms": round(rp[0]["t_ovl_median_ms"], 4),
                                "reduction_pct": round(100.0 * (1.0 - rp[3]["t_ovl_median_ms"] / rp[3]["t_seq_median_ms"]), 3),
                                "reduction_pct_normal_priority": round(
                                    100.0 * (1.0 - rp[0]["t_ovl_median_ms"] / rp[3]["t_seq_median_ms"]), 3),
                                "note": "medians"})
                pads.append(row)
            if pads:
                rec["extra_pads"] = pads
            rec["tuned"] = tuned(occ, wc, A, B, C, comm, args.steps)
            rec["roofline"] = roofline(wc, rc, "occ_gemm variant %d" % pc["kernel_id"], "kn")
            if not args.no_cpu_baseline:
                rec["cpu_baseline"] = cpu_baseline(wc, A, B, C, comm, args.config_cpu_budget, "kn")
            configs[name] = rec
        del A, B, C, comm
        torch.cuda.empty_cache()
    if configs:
        line["configs"] = configs
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
