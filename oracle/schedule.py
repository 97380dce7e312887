"""Schedule semantics of the overlap method (test infrastructure only).

Definitions taken from the paper:

* Section 3.2 -- two streams per device; the collective of iteration ``i``
  waits on an event recorded after the GEMM of iteration ``i``; later GEMMs
  may run while earlier collectives are still running.  Each stream executes
  its kernels in issue order.
* Section 3.3 -- the only required ordering is ``K_g^i -> K_c^i``.
* Section 4.2 -- ``TimeRatio = t_overlap / t_sequential`` and the overlap rate,
  the fraction of communication time that runs concurrently with computation.

Intervals are ``(start, end)`` pairs in any common time unit.
"""


def time_ratio(t_overlap, t_sequential):
    """Section 4.2: overlapped makespan over sequential makespan."""
    if t_sequential <= 0:
        raise ValueError("t_sequential must be positive")
    return t_overlap / t_sequential


def sequential_makespan(t_g, t_c):
    """All kernels on one stream in the order G0 C0 G1 C1 ... (Fig. 1a)."""
    if len(t_g) != len(t_c):
        raise ValueError("one GEMM and one collective per iteration")
    return float(sum(t_g) + sum(t_c))


def overlapped_makespan(t_g, t_c):
    """Two-stream pipelined schedule of Section 3.2 assuming no interference.

    The compute stream runs G0, G1, ... back to back.  The comm stream runs
    C_i once both G_i (event dependency) and C_{i-1} (stream order) are done.
    The makespan is the end of the last collective.
    """
    if len(t_g) != len(t_c):
        raise ValueError("one GEMM and one collective per iteration")
    g_end = 0.0
    c_end = 0.0
    for tg, tc in zip(t_g, t_c):
        g_end = g_end + tg
        c_start = max(g_end, c_end)
        c_end = c_start + tc
    return max(g_end, c_end)


def _union(intervals):
    out = []
    for s, e in sorted((float(s), float(e)) for s, e in intervals if e > s):
        if out and s <= out[-1][1]:
            out[-1][1] = max(out[-1][1], e)
        else:
            out.append([s, e])
    return out


def _length(intervals):
    return sum(e - s for s, e in intervals)


def overlap_rate(comp_intervals, comm_intervals):
    """Section 4.2: |union(comm) intersect union(comp)| / |union(comm)|."""
    comm = _union(comm_intervals)
    comp = _union(comp_intervals)
    total = _length(comm)
    if total == 0:
        return 0.0
    both = 0.0
    i = j = 0
    while i < len(comm) and j < len(comp):
        s = max(comm[i][0], comp[j][0])
        e = min(comm[i][1], comp[j][1])
        if e > s:
            both += e - s
        if comm[i][1] < comp[j][1]:
            i += 1
        else:
            j += 1
    return both / total


def dependency_violations(gemm_intervals, comm_intervals, sequential=False):
    """Orderings the schedule requires that a measured trace breaks.

    Always: end(G_i) <= start(C_i) (Section 3.3) and in-order execution on the
    compute stream and on the comm stream.  ``sequential=True`` additionally
    requires the single-stream order G0 C0 G1 C1 ... with no two kernels
    overlapping.  Returns a list of human-readable violations (empty = valid).
    """
    bad = []
    n = len(gemm_intervals)
    if len(comm_intervals) != n:
        return ["%d GEMMs but %d collectives" % (n, len(comm_intervals))]
    for i in range(n):
        if gemm_intervals[i][1] > comm_intervals[i][0]:
            bad.append("C%d starts before G%d ends" % (i, i))
        if i and gemm_intervals[i][0] < gemm_intervals[i - 1][1]:
            bad.append("G%d starts before G%d ends" % (i, i - 1))
        if i and comm_intervals[i][0] < comm_intervals[i - 1][1]:
            bad.append("C%d starts before C%d ends" % (i, i - 1))
        if sequential and i and gemm_intervals[i][0] < comm_intervals[i - 1][1]:
            bad.append("G%d starts before C%d ends (sequential)" % (i, i - 1))
    return bad
