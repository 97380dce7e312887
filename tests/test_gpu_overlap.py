"""The two-stream launcher: results, schedule semantics and timing sanity.

Section 3.3: overlap keeps the dependency K_g^i -> K_c^i and therefore the
results; the outputs after run_overlap must be bit-identical to one plain
occ_gemm and one plain share_* call, for every pad, priority and dependency
kind.  The kernel timeline recorded by the library must respect the
schedule's orderings (checked with the oracle's definitions), the
overlapped schedule must actually overlap (overlap rate, co-resident
workgroups of K_c^i and K_g^{i+1}, a makespan below the sequential one), and
the makespans must satisfy the bounds the schedule implies.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import schedule
from paper_2606_09200_amd import binding as occ
from paper_2606_09200_amd import inputs
from paper_2606_09200_amd import trace
from gpu_common import DEV, assert_gemm_close, bf16_bits

pytestmark = pytest.mark.gpu

DEPS = ("event", "counter")


def reduce_setup(M=512, N=512, K=512, nchunks=4, length=1 << 20):
    """GEMM operands with B stored K x N (occ_gemm's layout), C, chunks, out."""
    A, Bt = inputs.gemm_operands(M, N, K, seed=0, device=DEV)
    C = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    chunks = inputs.reduce_chunks(nchunks, length, seed=1, device=DEV)
    out = torch.empty(length, device=DEV)
    return A, Bt.t().contiguous(), C, chunks, out


def timeline_intervals(tl, n):
    t = tl.cpu().numpy().astype(np.int64).reshape(n, 4)
    g = [(int(r[0]), int(r[1])) for r in t]
    c = [(int(r[2]), int(r[3])) for r in t]
    return g, c


def check_reduce(C, out, A, B, chunks, M, N, K, what):
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), M, N, K, b_layout="kn")
    assert_gemm_close(bf16_bits(C), ref, 1.0, 1.0, K, what)
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32)), what


@pytest.mark.parametrize("dep", DEPS)
@pytest.mark.parametrize("pad,prio", [(0, 0), (0, 3), (64 << 10, 0), (64 << 10, 3)])
def test_overlap_results_match_plain_calls(pad, prio, dep):
    A, B, C, chunks, out = reduce_setup()
    C_ref = torch.empty_like(C)
    out_ref = torch.empty_like(out)
    occ.occ_gemm(A, B, C_ref)
    occ.share_reduce(chunks, out_ref)
    torch.cuda.synchronize()
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, lds_bytes=pad, comm_priority=prio,
                        n_iter=4, reps=2, warmup=1, dep=dep)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    assert torch.equal(out.view(torch.int32), out_ref.view(torch.int32))
    assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0 and r["t_gemm_ms"] > 0 and r["t_comm_ms"] > 0
    check_reduce(C, out, A, B, chunks, 512, 512, 512, "overlap %s" % dep)


@pytest.mark.parametrize("dep", DEPS)
def test_overlap_waits_for_the_callers_stream(dep):
    """Inputs still being written on the caller's (torch's) stream when
    run_overlap is called: the launcher's streams start after that work."""
    M = N = K = 1024
    A, B, C, chunks, out = reduce_setup(M, N, K, 4, 1 << 22)
    C_ref, out_ref = torch.empty_like(C), torch.empty_like(out)
    occ.occ_gemm(A, B, C_ref)
    occ.share_reduce(chunks, out_ref)
    A_in = torch.full_like(A, float("nan"))
    ch_in = torch.full_like(chunks, float("nan"))
    big = torch.empty(1 << 28, device=DEV)            # 1 GiB
    torch.cuda.synchronize()
    for _ in range(20):                               # several ms of queued work first
        big.fill_(1.0)
    A_in.copy_(A)
    ch_in.copy_(chunks)
    # issued with no host synchronisation since the fills and copies
    occ.run_overlap(A_in, B, C, bufs=ch_in, out=out, n_iter=2, reps=1, warmup=0, dep=dep)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    assert torch.equal(out.view(torch.int32), out_ref.view(torch.int32))


@pytest.mark.parametrize("dep", DEPS)
def test_overlap_skinny_gemm_matches_plain_calls_and_traces(dep):
    # decode-like M <= 16: the skinny K x N kernel (automatic choice) inside
    # both schedules, with every workgroup traced
    n, M, N, K = 3, 16, 1160, 2048
    A, Bt = inputs.gemm_operands(M, N, K, seed=5, device=DEV)
    B = Bt.t().contiguous()
    C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    C_ref = torch.empty_like(C)
    chunks = inputs.reduce_chunks(4, 1 << 20, seed=1, device=DEV)
    out = torch.empty(1 << 20, device=DEV)
    occ.occ_gemm(A, B, C_ref)
    plan = occ.occ_gemm_plan_query(M, N, K)
    assert plan["kernel_id"] == 33
    cap = 4096
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * cap, dtype=torch.int32, device=DEV)
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, comm_priority=0, n_iter=n,
                        reps=1, warmup=0, comm_wgs=32, wg_trace=wt, dep=dep)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), M, N, K, b_layout="kn")
    assert_gemm_close(bf16_bits(C), ref, 1.0, 1.0, K, "overlap skinny C")
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32))
    assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0
    recs = occ.decode_wg_trace(wt)
    assert int(wt[0]) == n * (plan["grid"] + 32) <= cap
    for i in range(n):
        g = [x for x in recs if x["tag"] == 2 * i]
        c = [x for x in recs if x["tag"] == 2 * i + 1]
        assert sorted(x["block"] for x in g) == list(range(plan["grid"]))
        assert min(x["t0"] for x in c) >= max(x["t1"] for x in g)


def test_overlap_bt_layout_matches_plain_calls():
    # the schedule with B stored N x K (occ_gemm_bt's layout)
    A, B, C, chunks, out = reduce_setup(M=520, N=264, K=200)
    Bt = B.t().contiguous()
    C_ref = torch.empty_like(C)
    occ.occ_gemm_bt(A, Bt, C_ref)
    torch.cuda.synchronize()
    for dep in DEPS:
        C.fill_(float("nan"))
        r = occ.run_overlap(A, Bt, C, bufs=chunks, out=out, b_layout="nk", comm_priority=0,
                            n_iter=3, reps=2, warmup=1, dep=dep)
        torch.cuda.synchronize()
        assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16)), dep
        assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0
    check_reduce(C, out, A, B, chunks, 520, 264, 200, "overlap bt")
    with pytest.raises(occ.OccError):                   # a variant that reads K x N
        occ.run_overlap(A, Bt, C, bufs=chunks, out=out, b_layout="nk", gemm_variant=32,
                        n_iter=1, reps=1, warmup=0)
    with pytest.raises(occ.OccError):                   # and the reverse
        occ.run_overlap(A, B, C, bufs=chunks, out=out, gemm_variant=16, n_iter=1, reps=1, warmup=0)


@pytest.mark.parametrize("dep", DEPS)
def test_overlap_permute_results_match_plain_calls(dep):
    A, Bt = inputs.gemm_operands(1024, 768, 512, seed=0, device=DEV)
    B = Bt.t().contiguous()
    C = torch.empty((1024, 768), device=DEV, dtype=torch.bfloat16)
    src = inputs.permute_payload(64, 1 << 16, seed=2, device=DEV)
    dst = torch.empty_like(src)
    perm = inputs.chunk_permutation(64, seed=3)
    r = occ.run_overlap(A, B, C, src=src, dst=dst, perm=perm, chunk_bytes=1 << 16, n_iter=3,
                        reps=2, warmup=1, dep=dep)
    torch.cuda.synchronize()
    want = oracle.permute_chunks(src.cpu().numpy(), perm.numpy(), 1 << 16)
    assert np.array_equal(dst.cpu().numpy(), want)
    assert r["t_ovl_ms"] > 0


@pytest.mark.parametrize("dep", DEPS)
def test_overlap_timeline_respects_schedule_and_overlaps(dep):
    """Mid size (2048 x 2048 x 4096 GEMM with an 8 x 2^22 chunk sum): the
    recorded kernel intervals keep K_g^i -> K_c^i and stream order, the
    collectives overlap the GEMMs (overlap rate > 0, at most (n-1)/n), and
    some workgroup of K_c^i shares a CU, in time, with a workgroup of
    K_g^{i+1}.  A serialised "overlap" fails all three."""
    n = 6
    A, B, C, chunks, out = reduce_setup(M=2048, N=2048, K=4096, nchunks=8, length=1 << 22)
    tl = torch.zeros(4 * n, dtype=torch.int64, device=DEV)
    cap = 16384
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * cap, dtype=torch.int32, device=DEV)
    occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=n, reps=1, warmup=1, timeline=tl, wg_trace=wt,
                    comm_priority=0, dep=dep)
    torch.cuda.synchronize()
    g, c = timeline_intervals(tl, n)
    assert all(e > s for s, e in g + c)
    assert schedule.dependency_violations(g, c) == []
    rate = schedule.overlap_rate(g, c)
    # the last collective starts after the last GEMM ended, so it never
    # overlaps: at most 1 - t(C_{n-1}) / sum t(C_i) ((n-1)/n for equal lengths)
    dur = [e - s for s, e in c]
    assert 0.2 < rate <= 1.0 - dur[-1] / sum(dur) + 1e-9, rate
    assert trace.overlap_rate(g, c) == pytest.approx(rate)
    recs = occ.decode_wg_trace(wt)
    assert int(wt[0]) <= cap
    pairs = 0
    for i in range(n - 1):
        ci = [x for x in recs if x["tag"] == 2 * i + 1]
        gn = [x for x in recs if x["tag"] == 2 * (i + 1)]
        gcu = {}
        for x in gn:
            gcu.setdefault(trace._cu_key(x), []).append((x["t0"], x["t1"]))
        for x in ci:
            for s, e in gcu.get(trace._cu_key(x), ()):
                if s < x["t1"] and x["t0"] < e:
                    pairs += 1
                    break
    assert pairs > 0


@pytest.mark.parametrize("dep", DEPS)
def test_makespan_bounds(dep):
    n = 8
    A, B, C, chunks, out = reduce_setup(M=2048, N=2048, K=4096, nchunks=8, length=1 << 23)
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=n, reps=3, warmup=2, comm_priority=0, dep=dep)
    tg, tc = r["t_gemm_ms"], r["t_comm_ms"]
    # sequential ~ n (t_g + t_c); the overlapped schedule is no faster than
    # its ideal n max + min (less a little noise) and, overlapping, shorter
    # than running everything back to back
    assert r["t_seq_ms"] == pytest.approx(n * (tg + tc), rel=0.25)
    assert r["t_ovl_ms"] >= 0.9 * (n * max(tg, tc) + min(tg, tc))
    assert r["t_ovl_ms"] < r["t_seq_ms"], r
    assert r["reduction_pct"] == pytest.approx(100 * (1 - r["t_ovl_ms"] / r["t_seq_ms"]))


def test_counter_dependency_cheaper_than_events_when_launch_bound():
    """The 512^3 GEMM + 4 x 2^20 chunk sum of the tiny workload: with the
    event per iteration the overlapped schedule is bound by host issue time;
    the device counter removes the two runtime calls per iteration."""
    A, B, C, chunks, out = reduce_setup()
    r_ev = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=10, reps=20, warmup=5,
                           flags=occ.OCC_RUN_OVL, dep="event")
    r_ct = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=10, reps=20, warmup=5,
                           flags=occ.OCC_RUN_OVL, dep="counter")
    assert r_ct["t_ovl_median_ms"] < r_ev["t_ovl_median_ms"], (r_ct, r_ev)


def test_counter_dependency_rejects_what_it_cannot_run():
    A, B, C, chunks, out = reduce_setup()
    cus = occ.occ_gemm_plan_query(512, 512, 512)["num_cus"]
    with pytest.raises(occ.OccError) as e:              # more than one comm workgroup per CU
        occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=2, reps=1, warmup=0, comm_wgs=cus + 1,
                        dep="counter")
    assert e.value.status == occ.OCC_EINVAL
    with pytest.raises(occ.OccError) as e:              # counters for at most 1024 iterations
        occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=1025, reps=1, warmup=0, dep="counter")
    assert e.value.status == occ.OCC_EINVAL
    # still usable afterwards (the counters were never touched)
    occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=2, reps=1, warmup=0, dep="counter")


def test_plan_reports_occupancy_shaping():
    r0 = occ.occ_gemm_plan_query(8192, 8192, 8192, 0, 37)
    r1 = occ.occ_gemm_plan_query(8192, 8192, 8192, 96 << 10, 37)
    assert r0["wg_per_cu"] > r1["wg_per_cu"] >= 1


def test_overlap_tune_picks_a_candidate_and_keeps_results():
    A, B, C, chunks, out = reduce_setup(M=2048, N=2048, K=4096, nchunks=8, length=1 << 23)
    knobs, r, prefer_seq = occ.occ_overlap_tune(A, B, C, bufs=chunks, out=out, n_iter=6, reps=3,
                                                warmup=1, tune_reps=2)
    torch.cuda.synchronize()
    assert knobs["comm_priority"] in (0, 3)
    cus = occ.occ_gemm_plan_query(2048, 2048, 4096)["num_cus"]
    assert knobs["comm_wgs"] in (0, 2 * cus, cus // 4)
    assert knobs["gemm_grid"] in (0, cus)
    assert knobs["dep"] in DEPS and not (knobs["dep"] == "counter" and knobs["comm_wgs"] > cus)
    assert r["t_ovl_ms"] > 0 and r["t_seq_ms"] > 0
    assert prefer_seq == (r["t_ovl_median_ms"] > r["t_seq_median_ms"])
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), 2048, 2048, 4096, b_layout="kn", rows=(0, 64),
                           cols=(1984, 2048))
    assert_gemm_close(bf16_bits(C)[0:64, 1984:2048], ref, 1.0, 1.0, 4096, "tuned C")
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32))


@pytest.mark.parametrize("kind", ["reduce", "permute"])
def test_graph_replays_match_eager(kind):
    """OCC_RUN_GRAPH captures both schedules once and replays them (warmup +
    reps times per call); outputs must equal the eager results after every
    call, with eager work (refilling the outputs) between the calls.  Graphs
    keep the event dependency: the counter is refused with them."""
    A, Bt = inputs.gemm_operands(768, 640, 512, seed=0, device=DEV)
    B = Bt.t().contiguous()
    C_ref = torch.empty((768, 640), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm(A, B, C_ref)
    if kind == "reduce":
        chunks = inputs.reduce_chunks(4, 1 << 18, seed=1, device=DEV)
        ref = torch.empty(1 << 18, device=DEV)
        occ.share_reduce(chunks, ref)
        comm = dict(bufs=chunks, out=torch.empty_like(ref))
        outk = "out"
    else:
        src = inputs.permute_payload(16, 1 << 14, seed=2, device=DEV)
        perm = inputs.chunk_permutation(16, seed=3)
        ref = torch.empty_like(src)
        occ.share_permute(src, ref, perm, 1 << 14)
        comm = dict(src=src, dst=torch.empty_like(src), perm=perm, chunk_bytes=1 << 14)
        outk = "dst"
    torch.cuda.synchronize()
    C = torch.empty_like(C_ref)
    for call in range(3):
        C.fill_(float("nan"))
        comm[outk].fill_(7)
        torch.cuda.synchronize()
        r = occ.run_overlap(A, B, C, n_iter=3, reps=2, warmup=1 + call,
                            flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL | occ.OCC_RUN_GRAPH, **comm)
        torch.cuda.synchronize()
        assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0
        assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16)), call
        assert torch.equal(comm[outk].view(torch.uint8), ref.view(torch.uint8)), call
    with pytest.raises(occ.OccError) as e:
        occ.run_overlap(A, B, C, n_iter=3, reps=1, warmup=0, dep="counter",
                        flags=occ.OCC_RUN_OVL | occ.OCC_RUN_GRAPH, **comm)
    assert e.value.status == occ.OCC_EINVAL


def test_wg_trace_records_every_workgroup():
    """One record per workgroup of every kernel of the traced pass, tagged
    with its iteration and kind, on a real CU and XCD, with an engine clock
    (cycles over elapsed 10 ns ticks) in the chip's range."""
    n = 3
    A, B, C, chunks, out = reduce_setup(M=2048, N=2048, K=2048, nchunks=4, length=1 << 22)
    cap = 8192
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * cap, dtype=torch.int32, device=DEV)
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=n, reps=1, warmup=0, comm_wgs=64,
                        wg_trace=wt)
    torch.cuda.synchronize()
    grid = occ.occ_gemm_plan_query(2048, 2048, 2048)["grid"]
    assert r["comm_wgs"] == 64
    assert int(wt[0]) == n * (grid + 64) <= cap
    recs = occ.decode_wg_trace(wt)
    for i in range(n):
        g = [x for x in recs if x["tag"] == 2 * i]
        c = [x for x in recs if x["tag"] == 2 * i + 1]
        assert len(g) == grid and sorted(x["block"] for x in g) == list(range(grid))
        assert len(c) == 64 and sorted(x["block"] for x in c) == list(range(64))
        assert all(x["kind"] == "gemm" for x in g) and all(x["kind"] == "comm" for x in c)
        # the collective of iteration i starts after the GEMM of iteration i ended
        assert min(x["t0"] for x in c) >= max(x["t1"] for x in g)
    assert all(x["t1"] >= x["t0"] and x["xcc"] < 8 for x in recs)
    ticks = sum(x["t1"] - x["t0"] for x in recs)
    cycles = sum(x["cycles"] for x in recs)
    ghz = cycles / (ticks * 10.0)
    assert 0.5 < ghz < 3.0, ghz


@pytest.mark.parametrize("kind", ["reduce", "reduce8", "permute"])
def test_paced_collective_keeps_results_and_rate(kind):
    """comm_rate_gbs paces the overlapped schedule's collective: results stay
    bit-identical, the sequential schedule stays unpaced, and the overlapped
    makespan is at least the paced transfer time of its n collectives."""
    n = 2
    A, Bt = inputs.gemm_operands(512, 512, 512, seed=0, device=DEV)
    B = Bt.t().contiguous()
    C = torch.empty((512, 512), device=DEV, dtype=torch.bfloat16)
    if kind.startswith("reduce"):
        # 4 and 8 chunks run instantiations with different positions per trip
        nch, length = (4, 1 << 20) if kind == "reduce" else (8, 1 << 19)
        chunks = inputs.reduce_chunks(nch, length, seed=1, device=DEV)
        ref = torch.empty(length, device=DEV)
        occ.share_reduce(chunks, ref)
        comm = dict(bufs=chunks, out=torch.empty_like(ref), comm_wgs=16)
        outk, nbytes, rate = "out", (nch + 1) * 4 * length, 20.0
    else:
        src = inputs.permute_payload(16, 1 << 16, seed=2, device=DEV)
        perm = inputs.chunk_permutation(16, seed=3)
        ref = torch.empty_like(src)
        occ.share_permute(src, ref, perm, 1 << 16)
        comm = dict(src=src, dst=torch.empty_like(src), perm=perm, chunk_bytes=1 << 16, comm_wgs=4)
        outk, nbytes, rate = "dst", 2 * 16 * (1 << 16), 10.0
    torch.cuda.synchronize()
    r = occ.run_overlap(A, B, C, n_iter=n, reps=2, warmup=1, comm_priority=0, comm_rate_gbs=rate, **comm)
    torch.cuda.synchronize()
    assert torch.equal(comm[outk].view(torch.uint8), ref.view(torch.uint8))
    paced_ms = nbytes / (rate * 1e9) * 1e3
    assert 0.8 * n * paced_ms <= r["t_ovl_ms"] <= 2.0 * n * paced_ms + r["t_seq_ms"], (r, paced_ms)
    assert r["t_comm_ms"] < 0.5 * paced_ms and r["t_seq_ms"] < r["t_ovl_ms"], r


def test_makespan_statistics():
    A, B, C, chunks, out = reduce_setup(M=1024, N=1024, K=1024, nchunks=4, length=1 << 20)
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=4, reps=7, warmup=1)
    for k in ("seq", "ovl"):
        mean, med, lo, sd = r["t_%s_ms" % k], r["t_%s_median_ms" % k], r["t_%s_min_ms" % k], r["t_%s_std_ms" % k]
        assert 0 < lo <= med and lo <= mean and sd >= 0
        assert mean - lo <= 3 * sd * 7 ** 0.5 + 1e-9       # min lies within the sample's spread
    r1 = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=2, reps=1, warmup=0)
    assert r1["t_seq_std_ms"] == 0 and r1["t_seq_median_ms"] == pytest.approx(r1["t_seq_ms"])
    assert r1["t_ovl_median_ms"] == pytest.approx(r1["t_ovl_ms"]) == r1["t_ovl_min_ms"]


def test_pace_all_paces_every_schedule():
    """OCC_RUN_PACE_ALL: the sequential schedule and the isolated timing run
    the collective paced too (link-bound emulation); results unchanged."""
    A, B, C, chunks, out = reduce_setup()
    ref = torch.empty_like(out)
    occ.share_reduce(chunks, ref)
    rate = 20.0
    paced_ms = 5 * 4 * (1 << 20) / (rate * 1e9) * 1e3
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, comm_wgs=16, comm_priority=0, n_iter=2, reps=1,
                        warmup=1, comm_rate_gbs=rate, flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL |
                        occ.OCC_RUN_ISO | occ.OCC_RUN_PACE_ALL)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    assert r["t_comm_ms"] >= 0.8 * paced_ms, r
    assert r["t_seq_ms"] >= 0.8 * 2 * paced_ms and r["t_ovl_ms"] >= 0.8 * 2 * paced_ms, r


@pytest.mark.parametrize("dep", DEPS)
@pytest.mark.parametrize("flags", [occ.OCC_RUN_OVL, occ.OCC_RUN_SEQ, occ.OCC_RUN_OVL | occ.OCC_RUN_GRAPH, 0])
def test_overlap_collective_consumes_each_iterations_gemm_output(flags, dep):
    # C holds one output per iteration, poisoned with NaN beforehand: every
    # C_i must be the GEMM's result and the last collective's output the
    # fixed-order sum of C_{n-1} and the peer chunks, i.e. each collective
    # read its own iteration's output after that GEMM wrote it (through the
    # event, or the counter's release / acquire)
    n_iter, M, N, K = 4, 520, 264, 136
    A, Bt = inputs.gemm_operands(M, N, K, seed=3, device=DEV)
    B = Bt.t().contiguous()
    C = torch.full((n_iter, M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    peers = inputs.reduce_chunks(3, M * N, seed=4, device=DEV)
    out = torch.full((M * N,), float("nan"), device=DEV)
    C_ref = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm(A, B, C_ref)
    if dep == "counter" and flags & occ.OCC_RUN_GRAPH:      # graphs keep the event
        with pytest.raises(occ.OccError):
            occ.run_overlap(A, B, C, bufs=peers, out=out, reduce_own=True, n_iter=n_iter, reps=1,
                            warmup=0, flags=flags, dep=dep)
        return
    r = occ.run_overlap(A, B, C, bufs=peers, out=out, reduce_own=True, n_iter=n_iter, reps=1, warmup=0,
                        flags=flags, comm_priority=0, dep=dep)
    torch.cuda.synchronize()
    for i in range(n_iter):
        assert torch.equal(C[i].view(torch.int16), C_ref.view(torch.int16)), i
    ref = oracle.chunk_sum_own_f32(C[-1].cpu(), peers.cpu().numpy())
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    if flags & occ.OCC_RUN_OVL or flags == 0:
        assert r["t_ovl_ms"] > 0
    if flags & occ.OCC_RUN_SEQ or flags == 0:
        assert r["t_seq_ms"] > 0


@pytest.mark.parametrize("dep", DEPS)
def test_overlap_reduce_own_no_peers_and_timeline(dep):
    n_iter, M, N, K = 3, 256, 256, 512
    A, Bt = inputs.gemm_operands(M, N, K, seed=5, device=DEV)
    B = Bt.t().contiguous()
    C = torch.zeros((n_iter, M, N), device=DEV, dtype=torch.bfloat16)
    out = torch.empty(M * N, device=DEV)
    tl = torch.zeros(4 * n_iter, dtype=torch.int64, device=DEV)
    occ.run_overlap(A, B, C, bufs=None, out=out, reduce_own=True, n_iter=n_iter, reps=1, warmup=0,
                    flags=occ.OCC_RUN_OVL, timeline=tl, dep=dep)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          C[-1].view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1).astype(np.uint32) << 16)
    g, c = timeline_intervals(tl, n_iter)
    assert schedule.dependency_violations(g, c) == []


# ------------------------------------------------------- occ_overlap_enqueue
@pytest.mark.parametrize("kind", ["reduce", "permute", "own"])
def test_overlap_enqueue_matches_plain_calls(kind):
    """The enqueued overlapped schedule (no events, device counters in a
    caller workspace) computes what the plain calls compute, reports no
    timeout, and leaves its workspace zeroed for the next schedule, which
    runs on the same workspace with fewer iterations."""
    M, N, K = 520, 264, 136
    A, Bt = inputs.gemm_operands(M, N, K, seed=3, device=DEV)
    B = Bt.t().contiguous()
    s1 = torch.cuda.Stream()
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    for n_iter in (6, 3):
        nbytes = occ.occ_overlap_workspace_bytes(n_iter)
        ws = torch.zeros(nbytes // 4, dtype=torch.int32, device=DEV) if n_iter == 6 else ws
        C_ref = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
        occ.occ_gemm(A, B, C_ref)
        if kind == "own":
            C = torch.full((n_iter, M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
            peers = inputs.reduce_chunks(3, M * N, seed=4, device=DEV)
            comm = dict(bufs=peers, out=torch.full((M * N,), float("nan"), device=DEV), reduce_own=True)
        else:
            C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
            if kind == "reduce":
                chunks = inputs.reduce_chunks(4, 1 << 18, seed=1, device=DEV)
                comm = dict(bufs=chunks, out=torch.full((1 << 18,), float("nan"), device=DEV))
            else:
                src = inputs.permute_payload(16, 1 << 14, seed=2, device=DEV)
                perm = inputs.chunk_permutation(16, seed=3)
                comm = dict(src=src, dst=torch.zeros_like(src), perm=perm, chunk_bytes=1 << 14)
        torch.cuda.synchronize()                      # both streams follow the inputs
        occ.occ_overlap_enqueue(A, B, C, workspace=ws, comm_stream=s1, err=err, n_iter=n_iter, **comm)
        torch.cuda.synchronize()
        assert int(err.item()) == 0
        assert int(ws.abs().sum().item()) == 0        # every counter back at zero
        if kind == "own":
            for i in range(n_iter):
                assert torch.equal(C[i].view(torch.int16), C_ref.view(torch.int16)), i
            ref = oracle.chunk_sum_own_f32(C[-1].cpu(), peers.cpu().numpy())
            assert np.array_equal(comm["out"].cpu().numpy().view(np.uint32), ref.view(np.uint32))
        else:
            assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
            if kind == "reduce":
                ref = oracle.chunk_sum_f32(chunks.cpu().numpy())
                assert np.array_equal(comm["out"].cpu().numpy().view(np.uint32), ref.view(np.uint32))
            else:
                want = oracle.permute_chunks(src.cpu().numpy(), perm.numpy(), 1 << 14)
                assert np.array_equal(comm["dst"].cpu().numpy(), want)


def test_overlap_enqueue_back_to_back_without_host_sync():
    """A serving loop: five schedules on one workspace, each one's GEMM stream
    ordered after the previous one's collectives by a stream event only, no
    host synchronisation in between (so a collective's counter reset and the
    next schedule's GEMM are ordered by the device alone).  Every output is
    right, no wait runs out, and the workspace ends at zero."""
    M, N, K = 520, 264, 136
    A, Bt = inputs.gemm_operands(M, N, K, seed=5, device=DEV)
    B = Bt.t().contiguous()
    C_ref = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm(A, B, C_ref)
    n_iter, rounds = 4, 5
    chunks = [inputs.reduce_chunks(4, 1 << 18, seed=10 + r, device=DEV) for r in range(rounds)]
    outs = [torch.full((1 << 18,), float("nan"), device=DEV) for _ in range(rounds)]
    Cs = [torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16) for _ in range(rounds)]
    ws = torch.zeros(occ.occ_overlap_workspace_bytes(n_iter) // 4, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    s0 = torch.cuda.current_stream()
    s1 = torch.cuda.Stream()
    torch.cuda.synchronize()
    for r in range(rounds):
        occ.occ_overlap_enqueue(A, B, Cs[r], workspace=ws, comm_stream=s1, err=err, n_iter=n_iter,
                                bufs=chunks[r], out=outs[r])
        done = torch.cuda.Event()
        done.record(s1)
        s0.wait_event(done)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    assert int(ws.abs().sum().item()) == 0
    for r in range(rounds):
        assert torch.equal(Cs[r].view(torch.int16), C_ref.view(torch.int16)), r
        ref = oracle.chunk_sum_f32(chunks[r].cpu().numpy())
        assert np.array_equal(outs[r].cpu().numpy().view(np.uint32), ref.view(np.uint32)), r


def test_overlap_enqueue_rejects_what_it_cannot_run():
    A, B, C, chunks, out = reduce_setup()
    s1 = torch.cuda.Stream()
    cus = occ.occ_gemm_plan_query(512, 512, 512)["num_cus"]
    ws = torch.zeros(occ.occ_overlap_workspace_bytes(4) // 4, dtype=torch.int32, device=DEV)
    with pytest.raises(occ.OccError) as e:            # more than one comm workgroup per CU
        occ.occ_overlap_enqueue(A, B, C, workspace=ws, comm_stream=s1, bufs=chunks, out=out, n_iter=4,
                                comm_wgs=cus + 1)
    assert e.value.status == occ.OCC_EINVAL
    with pytest.raises(occ.OccError) as e:            # workspace too short for 64 iterations
        occ.occ_overlap_enqueue(A, B, C, workspace=ws, comm_stream=s1, bufs=chunks, out=out, n_iter=64)
    assert e.value.status == occ.OCC_EINVAL
    torch.cuda.synchronize()
    assert int(ws.abs().sum().item()) == 0            # nothing was launched
