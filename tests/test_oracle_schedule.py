"""Pins the schedule definitions (Sections 3.2, 3.3 and 4.2) to closed forms."""
import pytest

from oracle import schedule


def test_time_ratio_definition():
    assert schedule.time_ratio(3.0, 10.0) == pytest.approx(0.3)
    with pytest.raises(ValueError):
        schedule.time_ratio(1.0, 0.0)


@pytest.mark.parametrize("tg,tc,n", [(5.0, 2.0, 10), (2.0, 5.0, 10), (3.0, 3.0, 4), (1.0, 0.5, 1)])
def test_overlapped_makespan_closed_form(tg, tc, n):
    # equal durations: n * max + min (the last collective cannot overlap)
    assert schedule.overlapped_makespan([tg] * n, [tc] * n) == pytest.approx(n * max(tg, tc) + min(tg, tc))
    assert schedule.sequential_makespan([tg] * n, [tc] * n) == pytest.approx(n * (tg + tc))


def test_overlapped_makespan_unequal_durations():
    # G: 0-4, 4-5, 5-11; C0 4-7, C1 7-9 (after C0), C2 11-12
    assert schedule.overlapped_makespan([4, 1, 6], [3, 2, 1]) == 12


def test_overlap_rate_examples():
    comp = [(0, 10), (10, 20)]
    comm = [(10, 14), (20, 24)]
    assert schedule.overlap_rate(comp, comm) == pytest.approx(0.5)
    assert schedule.overlap_rate([(0, 1)], [(2, 3)]) == 0.0
    assert schedule.overlap_rate([(0, 10)], [(2, 3), (4, 6)]) == 1.0
    assert schedule.overlap_rate([(0, 5), (3, 8)], [(6, 10)]) == pytest.approx(0.5)


def test_overlap_rate_bound_on_ideal_pipeline():
    # Section 4.2: the last collective waits for the last GEMM, so with equal
    # collective durations at most (n-1)/n of communication can overlap.
    for n in (2, 5, 10):
        tg, tc = 5.0, 2.0
        comp = [(i * tg, (i + 1) * tg) for i in range(n)]
        comm = [((i + 1) * tg, (i + 1) * tg + tc) for i in range(n)]
        assert schedule.overlap_rate(comp, comm) == pytest.approx((n - 1) / n)


def test_dependency_checks():
    g = [(0, 4), (4, 8)]
    ok = [(4, 6), (8, 9)]
    assert schedule.dependency_violations(g, ok) == []
    early = [(3, 6), (8, 9)]
    assert any("C0" in v for v in schedule.dependency_violations(g, early))
    assert schedule.dependency_violations(g, ok, sequential=True)  # G1 overlaps C0
    gs = [(0, 4), (6, 8)]
    assert schedule.dependency_violations(gs, ok := [(4, 6), (8, 9)], sequential=True) == []
