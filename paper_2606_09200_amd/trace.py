"""Host-side analysis of the kernel timeline and per-workgroup trace that
run_overlap records (occ_overlap_cfg.timeline / .wg_trace).

* ``intervals``      -- the timeline as GEMM and collective [start, end) lists;
* ``overlap_rate``   -- fraction of the collective's time during which a GEMM
                        kernel was also running (Section 4.2's overlap rate);
* ``coresidency``    -- fraction of collective workgroups that ran on a CU
                        while a GEMM workgroup ran on the same CU;
* ``interference``   -- GEMM workgroups split by whether a collective kernel
                        was running at the time: their mean lifetime and the
                        engine clock they ran at (cycles / elapsed time);
* ``residency``      -- achieved residency: the most workgroups of one kind
                        that ran at the same time on one CU.

Clock ticks are the GPU's constant 100 MHz clock (10 ns); cycles are
engine-clock cycles.
"""
import numpy as np

TICK_NS = 10.0


def intervals(timeline, n_iter):
    """timeline: 4*n_iter integers [g0 start, g0 end, c0 start, c0 end, ...]."""
    t = [int(x) for x in (timeline.tolist() if hasattr(timeline, "tolist") else timeline)]
    if len(t) < 4 * n_iter:
        raise ValueError("timeline holds %d entries, need %d" % (len(t), 4 * n_iter))
    g = [(t[4 * i], t[4 * i + 1]) for i in range(n_iter)]
    c = [(t[4 * i + 2], t[4 * i + 3]) for i in range(n_iter)]
    return g, c


def overlap_rate(g, c):
    """Time the collective kernels share with GEMM kernels over their total
    time; the kernels of one stream never overlap each other."""
    total = sum(e - s for s, e in c)
    if total <= 0:
        return 0.0
    both = sum(max(0, min(ce, ge) - max(cs, gs)) for cs, ce in c for gs, ge in g)
    return both / total


def _cu_key(r):
    return ((r["xcc"] * 8 + r["se"]) * 2 + r["sh"]) * 16 + r["cu"]


def coresidency(records):
    """Fraction of collective workgroups that shared a CU, in time, with a
    GEMM workgroup; None without collective records."""
    g = [(_cu_key(r), r["t0"], r["t1"]) for r in records if r["kind"] == "gemm"]
    c = [(_cu_key(r), r["t0"], r["t1"]) for r in records if r["kind"] == "comm"]
    if not c:
        return None
    if not g:
        return 0.0
    ga = np.array(g, dtype=np.int64)
    hit = 0
    for cu, s, e in c:
        m = (ga[:, 0] == cu) & (ga[:, 1] < e) & (ga[:, 2] > s)
        hit += bool(m.any())
    return hit / len(c)


def interference(records, comm_spans):
    """GEMM workgroups whose lifetime overlaps a collective kernel's span
    ("with_comm") against the others ("alone"): count, mean lifetime (us) and
    median engine clock (GHz).  comm_spans: [(start, end)] in ticks."""
    out = {}
    gem = [r for r in records if r["kind"] == "gemm" and r["t1"] > r["t0"]]
    spans = np.array(comm_spans, dtype=np.int64).reshape(-1, 2)
    for r in gem:
        r_conc = bool(((spans[:, 0] < r["t1"]) & (spans[:, 1] > r["t0"])).any()) if len(spans) else False
        key = "with_comm" if r_conc else "alone"
        d = out.setdefault(key, {"n": 0, "dur": [], "ghz": []})
        d["n"] += 1
        ticks = r["t1"] - r["t0"]
        d["dur"].append(ticks * TICK_NS / 1e3)
        if r.get("cycles", 0) > 0:
            d["ghz"].append(r["cycles"] / (ticks * TICK_NS))
    res = {}
    for k, d in out.items():
        res[k] = {"n": d["n"], "mean_us": round(float(np.mean(d["dur"])), 2),
                  "clock_ghz": round(float(np.median(d["ghz"])), 3) if d["ghz"] else None}
    return res


def residency(records, kind="gemm"):
    """Achieved residency of ``kind`` workgroups: for every CU the largest
    number of them alive at one instant (a workgroup ending at t does not
    overlap one starting at t).  Returns {"median": m, "max": x, "cus": n}
    over the CUs that ran any, or None."""
    per = {}
    for r in records:
        if r["kind"] == kind:
            per.setdefault(_cu_key(r), []).append((r["t0"], r["t1"]))
    if not per:
        return None
    peaks = []
    for ivs in per.values():
        ev = sorted([(t0, 1) for t0, _ in ivs] + [(t1, -1) for _, t1 in ivs], key=lambda e: (e[0], e[1]))
        cur = best = 0
        for _, d in ev:
            cur += d
            best = max(best, cur)
        peaks.append(best)
    return {"median": float(np.median(peaks)), "max": int(max(peaks)), "cus": len(peaks)}
