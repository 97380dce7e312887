"""Measure every workload configuration and the pad x priority sweep.

    python3 paper_2606_09200_amd/sweep.py --out results.md [--json results.jsonl]

For each point: sequential and overlapped makespans of 10 GEMM -> collective
iterations (Section 3.2; 5 timed repetitions after 2 warm-up, Section 4.1),
the reduction 100*(1 - TimeRatio) (Section 4.2), the isolated kernel times
with the GEMM's MFMA fraction and the comm kernel's HBM fraction, the GEMM's
resident workgroups per CU (Section 3.1), the overlap rate (Section 4.2) and
the fraction of comm workgroups that shared a CU with a running GEMM
workgroup, and the GEMM workgroups' mean lifetime and engine clock with and
without a collective running (from the per-workgroup trace).
"""
import argparse
import json
import os
import sys

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import numpy as np  # noqa: E402
import torch  # noqa: E402

from paper_2606_09200_amd import binding as occ  # noqa: E402
from paper_2606_09200_amd import inputs  # noqa: E402
from paper_2606_09200_amd import trace  # noqa: E402
from paper_2606_09200_amd.workloads import BLOCK_COUNTS, WORKLOADS  # noqa: E402

PEAK_TFLOPS = 2500.0
PEAK_GBS = 8000.0


def setup(w, dev, b_layout="kn"):
    A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_a=w.std_a, std_b=w.std_b,
                                 seed_b=w.seed_b, device=dev)
    B = Bt.t().contiguous() if b_layout == "kn" else Bt   # the same op(B) in the chosen layout
    del Bt
    if w.comm == "reduce_own":
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


# The tiles of the pad sweep and the thread-block-count study, per layout of
# B: the default tile (128 KiB of LDS: only small pads fit) and tiles small
# enough for the pad to set residency -- 128x256x32 (48 KiB, two per CU),
# 128x128x64 (96 KiB, three stages) and the paper's opt2 64x64x64 -- and the
# paper's two tiles (opt1 64x64x32, opt2 64x64x64).
SWEEP_VARIANTS = {"kn": (0, 38, 35, 37), "nk": (0, 25, 14, 7)}
BLOCK_VARIANTS = {"kn": (36, 37), "nk": (6, 7)}


def measure(w, A, B, C, comm, pad, prio, dev, reps=5, warmup=2, flags=0, **knobs):
    plan = occ.occ_gemm_plan_query(w.M, w.N, w.K, pad, knobs.get("gemm_variant", 0), knobs.get("gemm_grid", 0),
                                   b_layout=knobs.get("b_layout", "kn"))
    row = {"workload": w.name, "pad_kib": pad >> 10, "comm_priority": prio,
           "gemm_grid": plan["grid"],
           "gemm_variant": plan["kernel_id"], "gemm_tile_lds": plan["tile_lds_bytes"],
           "gemm_wg_per_cu": plan["wg_per_cu"] if plan["feasible"] else 0, "feasible": plan["feasible"]}
    if not plan["feasible"]:
        return row
    tl = torch.zeros(4 * w.n_iter, dtype=torch.int64, device=dev)
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * 60000, dtype=torch.int32, device=dev)
    r = occ.run_overlap(A, B, C, lds_bytes=pad, comm_priority=prio, n_iter=w.n_iter, reps=reps,
                        warmup=warmup, timeline=tl, wg_trace=wt, flags=flags, **knobs, **comm)
    tg, tc = r["t_gemm_ms"], r["t_comm_ms"]
    g_iv, c_iv = trace.intervals(tl.cpu(), w.n_iter)
    recs = occ.decode_wg_trace(wt)
    inter = trace.interference(recs, c_iv)
    row.update({
        "t_seq_ms": round(r["t_seq_ms"], 4), "t_ovl_ms": round(r["t_ovl_ms"], 4),
        "reduction_pct": round(r["reduction_pct"], 2),
        "time_ratio": round(r["t_ovl_ms"] / r["t_seq_ms"], 4),
        "ideal_ovl_ms": round(w.n_iter * max(tg, tc) + min(tg, tc), 4),
        "t_gemm_ms": round(tg, 4), "t_comm_ms": round(tc, 4),
        "gemm_tflops": round(w.gemm_flops / tg / 1e9, 1),
        "gemm_mfma_frac": round(w.gemm_flops / tg / 1e9 / PEAK_TFLOPS, 4),
        "gemm_hbm_frac": round(w.gemm_bytes / tg / 1e6 / PEAK_GBS, 4),
        "comm_gbs": round(w.comm_bytes / tc / 1e6, 1),
        "comm_hbm_frac": round(w.comm_bytes / tc / 1e6 / PEAK_GBS, 4),
        "comm_wgs": r["comm_wgs"],
        "overlap_rate": round(trace.overlap_rate(g_iv, c_iv), 4),
        "comm_ovl_us": round(sum(e - s for s, e in c_iv) / len(c_iv) * trace.TICK_NS / 1e3, 1),
        "comm_coresident": trace.coresidency(recs),
        "gemm_wg_per_cu_achieved": (trace.residency(recs) or {}).get("median"),
        "gemm_wg_us_alone": inter.get("alone", {}).get("mean_us"),
        "gemm_wg_us_with_comm": inter.get("with_comm", {}).get("mean_us"),
        "gemm_clock_ghz_alone": inter.get("alone", {}).get("clock_ghz"),
        "gemm_clock_ghz_with_comm": inter.get("with_comm", {}).get("clock_ghz"),
    })
    return row


def table(rows):
    cols = ["workload", "b_layout", "dep", "graph", "pace_all", "gemm_variant", "gemm_grid", "pad_kib", "comm_priority", "comm_wgs",
            "comm_rate_gbs", "gemm_wg_per_cu", "gemm_wg_per_cu_achieved", "t_seq_ms", "t_ovl_ms",
            "reduction_pct", "norm_time", "ideal_ovl_ms", "t_gemm_ms", "gemm_mfma_frac", "gemm_hbm_frac",
            "t_comm_ms", "comm_hbm_frac", "comm_ovl_us", "overlap_rate", "comm_coresident", "gemm_wg_us_alone",
            "gemm_wg_us_with_comm", "gemm_clock_ghz_alone", "gemm_clock_ghz_with_comm"]
    out = ["| " + " | ".join(cols) + " |", "|" + "---|" * len(cols)]
    for r in rows:
        out.append("| " + " | ".join("" if r.get(c) is None else
                                     ("%.3f" % r[c] if isinstance(r.get(c), float) and c == "comm_coresident" else str(r.get(c, "")))
                                     for c in cols) + " |")
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=None, help="markdown table to write")
    ap.add_argument("--json", default=None, help="JSON lines to write")
    ap.add_argument("--graph", action="store_true",
                    help="replay each schedule from a HIP graph (OCC_RUN_GRAPH)")
    ap.add_argument("--tune", action="store_true",
                    help="also run occ_overlap_tune per workload and report its choice")
    ap.add_argument("--workloads", default="tiny,cb,mb,a2a,sweep,blocks,paper_cb_ar,paper_mb_ar,"
                                           "paper_cb_a2a,paper_mb_a2a")
    ap.add_argument("--comm-wgs", default="0",
                    help="comma list of comm workgroup counts (0 = library default)")
    ap.add_argument("--rates", default="0",
                    help="comma list of comm bandwidth pacings in GB/s for the overlapped schedule (0 = off)")
    ap.add_argument("--priorities", default=None,
                    help="comma list of comm wave priorities (default: each workload's own)")
    ap.add_argument("--gemm-grids", default=None,
                    help="comma list of persistent GEMM grid caps to run each workload with "
                         "(0 = one workgroup per tile); the rows then show the engine clock "
                         "against the number of CUs the GEMM keeps busy")
    ap.add_argument("--b-layout", default="kn", choices=["kn", "nk"],
                    help="GEMM B stored K x N (occ_gemm) or N x K (occ_gemm_bt)")
    ap.add_argument("--dep", default="event", choices=["event", "counter"],
                    help="per-iteration dependency of the overlapped schedule")
    ap.add_argument("--pace-all", action="store_true",
                    help="apply --rates to every schedule (OCC_RUN_PACE_ALL): emulates a collective "
                         "whose time is set by inter-GPU links")
    a = ap.parse_args(argv)
    dev = "cuda:0"
    rows = []
    for name in a.workloads.split(","):
        w = WORKLOADS[name]
        A, B, C, comm = setup(w, dev, a.b_layout)
        if name == "blocks":
            # the paper's two tiles over the thread-block counts of its tile-size study
            points = [dict(gemm_variant=v, gemm_grid=x * x) for v in BLOCK_VARIANTS[a.b_layout] for x in BLOCK_COUNTS]
        elif name == "sweep":
            points = [dict(gemm_variant=v) for v in SWEEP_VARIANTS[a.b_layout]]
        elif a.gemm_grids:
            points = [dict(gemm_variant=0, gemm_grid=int(g)) for g in a.gemm_grids.split(",")]
        else:
            points = [dict(gemm_variant=0)]
        prios = [int(x) for x in a.priorities.split(",")] if a.priorities else list(w.priorities)
        extra = [dict(comm_wgs=int(cw), comm_rate_gbs=float(rt))
                 for cw in a.comm_wgs.split(",") for rt in a.rates.split(",")]
        for knobs in points:
            for ex in extra:
                base = {}
                for pad in w.pads:
                    for prio in prios:
                        fl = (occ.OCC_RUN_GRAPH if a.graph else 0) | (occ.OCC_RUN_PACE_ALL if a.pace_all else 0)
                        row = measure(w, A, B, C, comm, pad, prio, dev, flags=fl, b_layout=a.b_layout,
                                      dep=a.dep, **knobs, **ex)
                        row["b_layout"] = a.b_layout
                        row["dep"] = a.dep
                        row["graph"] = bool(a.graph)
                        row["pace_all"] = bool(a.pace_all)
                        row["comm_rate_gbs"] = ex["comm_rate_gbs"]
                        if prio == 0:
                            base[pad] = row.get("t_ovl_ms")
                        elif base.get(pad) and row.get("t_ovl_ms"):
                            row["norm_time"] = round(row["t_ovl_ms"] / base[pad], 4)
                        rows.append(row)
                        print(json.dumps(row), flush=True)
        if a.tune and name not in ("sweep", "blocks"):
            knobs, r, prefer_seq = occ.occ_overlap_tune(A, B, C, n_iter=w.n_iter, reps=5, warmup=2,
                                                        tune_reps=3, b_layout=a.b_layout, **comm)
            row = {"workload": w.name + " (tuned)", "gemm_variant": "auto", "gemm_grid": knobs["gemm_grid"],
                   "pad_kib": knobs["lds_bytes"] >> 10, "comm_priority": knobs["comm_priority"],
                   "comm_wgs": knobs["comm_wgs"], "dep": knobs["dep"], "t_seq_ms": round(r["t_seq_ms"], 4),
                   "t_ovl_ms": round(r["t_ovl_ms"], 4), "reduction_pct": round(r["reduction_pct"], 2),
                   "t_gemm_ms": round(r["t_gemm_ms"], 4), "t_comm_ms": round(r["t_comm_ms"], 4),
                   "gemm_wg_per_cu": r["gemm_wg_per_cu"], "prefer_sequential": prefer_seq}
            rows.append(row)
            print(json.dumps(row), flush=True)
        del A, B, C, comm
        torch.cuda.empty_cache()
    if a.json:
        with open(a.json, "w") as f:
            for r in rows:
                f.write(json.dumps(r) + "\n")
    if a.out:
        with open(a.out, "w") as f:
            f.write(table(rows) + "\n")
    return 0


if __name__ == "__main__":
    sys.exit(main())
