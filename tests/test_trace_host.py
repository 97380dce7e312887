"""Host-side trace analysis (paper_2606_09200_amd.trace) on synthetic records.

The overlap rate of Section 4.2 is checked against the oracle's definition
(union of collective intervals intersected with the union of GEMM intervals)
on random per-stream-disjoint timelines; co-residency and the interference
split are checked on hand-built workgroup records whose answers are known.
"""
import random

import pytest

from oracle import schedule
from paper_2606_09200_amd import trace


def disjoint(rng, n, t0=0):
    out, t = [], t0
    for _ in range(n):
        t += rng.randrange(0, 50)
        d = rng.randrange(1, 100)
        out.append((t, t + d))
        t += d
    return out


@pytest.mark.parametrize("seed", range(20))
def test_overlap_rate_matches_oracle(seed):
    rng = random.Random(seed)
    n = rng.randrange(1, 12)
    g, c = disjoint(rng, n), disjoint(rng, n, rng.randrange(0, 100))
    assert trace.overlap_rate(g, c) == pytest.approx(schedule.overlap_rate(g, c), abs=1e-12)


def test_intervals_layout_and_errors():
    g, c = trace.intervals([1, 5, 6, 9, 10, 20, 21, 30], 2)
    assert g == [(1, 5), (10, 20)] and c == [(6, 9), (21, 30)]
    with pytest.raises(ValueError):
        trace.intervals([1, 2, 3], 1)


def rec(kind, xcc, cu, t0, t1, cycles=0, se=0, sh=0):
    return {"kind": kind, "xcc": xcc, "se": se, "sh": sh, "cu": cu, "t0": t0, "t1": t1, "cycles": cycles}


def test_coresidency_counts_same_cu_in_time_only():
    recs = [rec("gemm", 0, 3, 0, 100), rec("gemm", 1, 3, 0, 100),
            rec("comm", 0, 3, 50, 60),      # same CU, inside -> hit
            rec("comm", 0, 4, 50, 60),      # other CU -> miss
            rec("comm", 1, 3, 100, 120),    # same CU, after the GEMM ended -> miss
            rec("comm", 2, 3, 10, 20),      # other XCD -> miss
            rec("comm", 0, 3, 10, 20, se=1)]  # other shader engine -> miss
    assert trace.coresidency(recs) == pytest.approx(1 / 5)
    assert trace.coresidency([rec("gemm", 0, 0, 0, 1)]) is None
    assert trace.coresidency([rec("comm", 0, 0, 0, 1)]) == 0.0


def test_interference_split_and_clock():
    # 10 ns ticks: 100 ticks = 1 us; 2000 cycles in 1 us = 2 GHz
    recs = [rec("gemm", 0, 0, 0, 100, cycles=2000),
            rec("gemm", 0, 1, 0, 100, cycles=1800),
            rec("gemm", 0, 2, 200, 500, cycles=6600),   # overlaps the span [250, 300)
            rec("comm", 0, 2, 250, 300, cycles=100)]
    out = trace.interference(recs, [(250, 300)])
    assert out["alone"]["n"] == 2 and out["alone"]["mean_us"] == pytest.approx(1.0)
    assert out["alone"]["clock_ghz"] == pytest.approx(1.9)
    assert out["with_comm"]["n"] == 1 and out["with_comm"]["mean_us"] == pytest.approx(3.0)
    assert out["with_comm"]["clock_ghz"] == pytest.approx(2.2)
    assert trace.interference(recs, []) ["alone"]["n"] == 3


def test_residency_counts_simultaneous_workgroups_per_cu():
    recs = [rec("gemm", 0, 0, 0, 10), rec("gemm", 0, 0, 5, 15), rec("gemm", 0, 0, 15, 20),  # peak 2
            rec("gemm", 0, 1, 0, 10), rec("gemm", 0, 1, 10, 20),                           # back to back: 1
            rec("gemm", 1, 0, 0, 10), rec("gemm", 1, 0, 1, 9), rec("gemm", 1, 0, 2, 8),   # peak 3
            rec("comm", 0, 0, 0, 100)]
    r = trace.residency(recs)
    assert r == {"median": 2.0, "max": 3, "cus": 3}
    assert trace.residency(recs, "comm") == {"median": 1.0, "max": 1, "cus": 1}
    assert trace.residency([], "gemm") is None
