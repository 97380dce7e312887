"""The two-stream launcher: results, schedule semantics and timing sanity.

Section 3.3: overlap keeps the dependency K_g^i -> K_c^i and therefore the
results; the outputs after run_overlap must be bit-identical to one plain
occ_gemm and one plain share_* call, for every pad and priority.  The kernel
timeline recorded by the library must respect the schedule's orderings
(checked with the oracle's definitions), and the makespans must satisfy the
bounds the schedule implies.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import schedule
from paper_2606_09200_amd import binding as occ
from paper_2606_09200_amd import inputs
from gpu_common import DEV, assert_gemm_close, bf16_bits

pytestmark = pytest.mark.gpu


def tiny_reduce_setup(M=512, N=512, K=512, nchunks=4, length=1 << 20):
    A, B = inputs.gemm_operands(M, N, K, seed=0, device=DEV)
    C = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    chunks = inputs.reduce_chunks(nchunks, length, seed=1, device=DEV)
    out = torch.empty(length, device=DEV)
    return A, B, C, chunks, out


def timeline_intervals(tl, n):
    t = tl.cpu().numpy().astype(np.int64).reshape(n, 4)
    g = [(int(r[0]), int(r[1])) for r in t]
    c = [(int(r[2]), int(r[3])) for r in t]
    return g, c


@pytest.mark.parametrize("pad,prio", [(0, 0), (0, 3), (64 << 10, 0), (64 << 10, 3)])
def test_overlap_results_match_plain_calls(pad, prio):
    A, B, C, chunks, out = tiny_reduce_setup()
    C_ref = torch.empty_like(C)
    out_ref = torch.empty_like(out)
    occ.occ_gemm(A, B, C_ref)
    occ.share_reduce(chunks, out_ref)
    torch.cuda.synchronize()
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, lds_bytes=pad, comm_priority=prio,
                        n_iter=4, reps=2, warmup=1)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    assert torch.equal(out.view(torch.int32), out_ref.view(torch.int32))
    assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0 and r["t_gemm_ms"] > 0 and r["t_comm_ms"] > 0
    # and both equal the oracle
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), 512, 512, 512)
    assert_gemm_close(bf16_bits(C), ref, 1.0, 1.0, 512, "overlap C")
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32))


@pytest.mark.parametrize("b_layout,variant", [("nk", 34), ("kn", 33)])
def test_overlap_skinny_gemm_matches_plain_calls_and_traces(b_layout, variant):
    # decode-like M <= 16: the LDS-staged skinny kernels (automatic choice)
    # inside both schedules, with every workgroup traced
    n, M, N, K = 3, 16, 1160, 2048
    A, B = inputs.gemm_operands(M, N, K, seed=5, device=DEV)
    Bx = B.t().contiguous() if b_layout == "kn" else B
    C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    C_ref = torch.empty_like(C)
    chunks = inputs.reduce_chunks(4, 1 << 20, seed=1, device=DEV)
    out = torch.empty(1 << 20, device=DEV)
    (occ.occ_gemm_kn if b_layout == "kn" else occ.occ_gemm)(A, Bx, C_ref)
    plan = occ.occ_gemm_plan_query(M, N, K, b_layout=b_layout)
    assert plan["kernel_id"] == variant
    cap = 4096
    wt = torch.zeros(4 + occ.WG_RECORD_WORDS * cap, dtype=torch.int32, device=DEV)
    r = occ.run_overlap(A, Bx, C, bufs=chunks, out=out, b_layout=b_layout, comm_priority=0, n_iter=n,
                        reps=1, warmup=0, comm_wgs=32, wg_trace=wt)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(Bx), M, N, K, b_layout=b_layout)
    assert_gemm_close(bf16_bits(C), ref, 1.0, 1.0, K, "overlap skinny %s C" % b_layout)
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32))
    assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0
    recs = occ.decode_wg_trace(wt)
    assert int(wt[0]) == n * (plan["grid"] + 32) <= cap
    for i in range(n):
        g = [x for x in recs if x["tag"] == 2 * i]
        assert sorted(x["block"] for x in g) == list(range(plan["grid"]))


def test_overlap_permute_results_match_plain_calls():
    A, B = inputs.gemm_operands(1024, 768, 512, seed=0, device=DEV)
    C = torch.empty((1024, 768), device=DEV, dtype=torch.bfloat16)
    src = inputs.permute_payload(64, 1 << 16, seed=2, device=DEV)
    dst = torch.empty_like(src)
    perm = inputs.chunk_permutation(64, seed=3)
    r = occ.run_overlap(A, B, C, src=src, dst=dst, perm=perm, chunk_bytes=1 << 16, n_iter=3,
                        reps=2, warmup=1)
    torch.cuda.synchronize()
    want = oracle.permute_chunks(src.cpu().numpy(), perm.numpy(), 1 << 16)
    assert np.array_equal(dst.cpu().numpy(), want)
    assert r["t_ovl_ms"] > 0


def test_overlap_timeline_respects_schedule():
    n = 6
    A, B, C, chunks, out = tiny_reduce_setup(M=2048, N=2048, K=2048, nchunks=8, length=1 << 22)
    tl = torch.zeros(4 * n, dtype=torch.int64, device=DEV)
    occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=n, reps=1, warmup=1, timeline=tl)
    torch.cuda.synchronize()
    g, c = timeline_intervals(tl, n)
    assert all(e > s for s, e in g + c)
    assert schedule.dependency_violations(g, c) == []
    rate = schedule.overlap_rate(g, c)
    assert 0.0 <= rate <= 1.0


def test_makespan_bounds():
    n = 8
    A, B, C, chunks, out = tiny_reduce_setup(M=2048, N=2048, K=4096, nchunks=8, length=1 << 23)
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, n_iter=n, reps=3, warmup=2)
    tg, tc = r["t_gemm_ms"], r["t_comm_ms"]
    # sequential ~ n (t_g + t_c); overlap can be no faster than the busier
    # stream alone and no slower than running everything back to back (+ slack)
    assert r["t_seq_ms"] == pytest.approx(n * (tg + tc), rel=0.25)
    assert r["t_ovl_ms"] >= 0.8 * n * max(tg, tc)
    assert r["t_ovl_ms"] <= 1.25 * r["t_seq_ms"]
    assert r["reduction_pct"] == pytest.approx(100 * (1 - r["t_ovl_ms"] / r["t_seq_ms"]))


def test_plan_reports_occupancy_shaping():
    r0 = occ.occ_gemm_plan_query(8192, 8192, 8192, 0, 5)
    r1 = occ.occ_gemm_plan_query(8192, 8192, 8192, 96 << 10, 5)
    assert r0["wg_per_cu"] >= r1["wg_per_cu"] >= 1


def test_overlap_tune_picks_a_candidate_and_keeps_results():
    A, B, C, chunks, out = tiny_reduce_setup(M=2048, N=2048, K=4096, nchunks=8, length=1 << 23)
    knobs, r, prefer_seq = occ.occ_overlap_tune(A, B, C, bufs=chunks, out=out, n_iter=6, reps=3,
                                                warmup=1, tune_reps=2)
    torch.cuda.synchronize()
    assert knobs["comm_priority"] in (0, 3)
    cus = occ.occ_gemm_plan_query(2048, 2048, 4096)["num_cus"]
    assert knobs["comm_wgs"] in (0, 2 * cus)
    assert knobs["gemm_grid"] in (0, cus)
    assert r["t_ovl_ms"] > 0 and r["t_seq_ms"] > 0
    assert prefer_seq == (r["t_ovl_ms"] > r["t_seq_ms"])
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), 2048, 2048, 4096, rows=(0, 64), cols=(1984, 2048))
    assert_gemm_close(bf16_bits(C)[0:64, 1984:2048], ref, 1.0, 1.0, 4096, "tuned C")
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32))


@pytest.mark.parametrize("kind", ["reduce", "permute"])
def test_graph_replays_match_eager(kind):
    """OCC_RUN_GRAPH captures both schedules once and replays them (warmup +
    reps times per call); outputs must equal the eager results after every
    call, with eager work (refilling the outputs) between the calls."""
    A, B = inputs.gemm_operands(768, 640, 512, seed=0, device=DEV)
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


def test_wg_trace_records_every_workgroup():
    """One record per workgroup of every kernel of the traced pass, tagged
    with its iteration and kind, on a real CU and XCD, with an engine clock
    (cycles over elapsed 10 ns ticks) in the chip's range."""
    n = 3
    A, B, C, chunks, out = tiny_reduce_setup(M=2048, N=2048, K=2048, nchunks=4, length=1 << 22)
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
    A, B = inputs.gemm_operands(512, 512, 512, seed=0, device=DEV)
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
    A, B, C, chunks, out = tiny_reduce_setup(M=1024, N=1024, K=1024, nchunks=4, length=1 << 20)
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
    A, B = inputs.gemm_operands(512, 512, 512, seed=0, device=DEV)
    C = torch.empty((512, 512), device=DEV, dtype=torch.bfloat16)
    chunks = inputs.reduce_chunks(4, 1 << 20, seed=1, device=DEV)
    ref = torch.empty(1 << 20, device=DEV)
    occ.share_reduce(chunks, ref)
    out = torch.empty_like(ref)
    rate = 20.0
    paced_ms = 5 * 4 * (1 << 20) / (rate * 1e9) * 1e3
    r = occ.run_overlap(A, B, C, bufs=chunks, out=out, comm_wgs=16, comm_priority=0, n_iter=2, reps=1,
                        warmup=1, comm_rate_gbs=rate, flags=occ.OCC_RUN_SEQ | occ.OCC_RUN_OVL |
                        occ.OCC_RUN_ISO | occ.OCC_RUN_PACE_ALL)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
    assert r["t_comm_ms"] >= 0.8 * paced_ms, r
    assert r["t_seq_ms"] >= 0.8 * 2 * paced_ms and r["t_ovl_ms"] >= 0.8 * 2 * paced_ms, r


def test_overlap_with_kn_b_matches_plain_calls():
    A, B, C, chunks, out = tiny_reduce_setup(M=520, N=264, K=200)
    Bkn = B.t().contiguous()
    C_ref = torch.empty_like(C)
    occ.occ_gemm_kn(A, Bkn, C_ref)
    torch.cuda.synchronize()
    r = occ.run_overlap(A, Bkn, C, bufs=chunks, out=out, b_layout="kn", comm_priority=0,
                        n_iter=3, reps=2, warmup=1)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    assert r["t_seq_ms"] > 0 and r["t_ovl_ms"] > 0
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(Bkn), 520, 264, 200, b_layout="kn")
    assert_gemm_close(bf16_bits(C), ref, 1.0, 1.0, 200, "overlap kn C")
    with pytest.raises(occ.OccError):                   # a variant that reads N x K
        occ.run_overlap(A, Bkn, C, bufs=chunks, out=out, b_layout="kn", gemm_variant=16,
                        n_iter=1, reps=1, warmup=0)


def test_overlap_tune_with_kn_b_keeps_results():
    A, B, C, chunks, out = tiny_reduce_setup(M=1024, N=1024, K=2048, nchunks=4, length=1 << 22)
    Bkn = B.t().contiguous()
    C_ref = torch.empty_like(C)
    occ.occ_gemm_kn(A, Bkn, C_ref)
    knobs, r, prefer_seq = occ.occ_overlap_tune(A, Bkn, C, bufs=chunks, out=out, n_iter=4, reps=2,
                                                warmup=1, tune_reps=1, b_layout="kn")
    torch.cuda.synchronize()
    assert r["t_ovl_ms"] > 0 and r["t_seq_ms"] > 0
    assert torch.equal(C.view(torch.int16), C_ref.view(torch.int16))
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          oracle.chunk_sum_f32(chunks.cpu().numpy()).view(np.uint32))


@pytest.mark.parametrize("flags", [occ.OCC_RUN_OVL, occ.OCC_RUN_SEQ, occ.OCC_RUN_OVL | occ.OCC_RUN_GRAPH, 0])
def test_overlap_collective_consumes_each_iterations_gemm_output(flags):
    # C holds one output per iteration, poisoned with NaN beforehand: every
    # C_i must be the GEMM's result and the last collective's output the
    # fixed-order sum of C_{n-1} and the peer chunks, i.e. each collective
    # read its own iteration's output after that GEMM wrote it
    n_iter, M, N, K = 4, 520, 264, 136
    A, B = inputs.gemm_operands(M, N, K, seed=3, device=DEV)
    C = torch.full((n_iter, M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    peers = inputs.reduce_chunks(3, M * N, seed=4, device=DEV)
    out = torch.full((M * N,), float("nan"), device=DEV)
    C_ref = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm(A, B, C_ref)
    r = occ.run_overlap(A, B, C, bufs=peers, out=out, reduce_own=True, n_iter=n_iter, reps=1, warmup=0,
                        flags=flags, comm_priority=0)
    torch.cuda.synchronize()
    for i in range(n_iter):
        assert torch.equal(C[i].view(torch.int16), C_ref.view(torch.int16)), i
    ref = oracle.chunk_sum_own_f32(C[-1].cpu(), peers.cpu().numpy())
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))
    if flags & occ.OCC_RUN_OVL or flags == 0:
        assert r["t_ovl_ms"] > 0
    if flags & occ.OCC_RUN_SEQ or flags == 0:
        assert r["t_seq_ms"] > 0


def test_overlap_reduce_own_no_peers_and_timeline():
    n_iter, M, N, K = 3, 256, 256, 512
    A, B = inputs.gemm_operands(M, N, K, seed=5, device=DEV)
    C = torch.zeros((n_iter, M, N), device=DEV, dtype=torch.bfloat16)
    out = torch.empty(M * N, device=DEV)
    tl = torch.zeros(4 * n_iter, dtype=torch.int64, device=DEV)
    occ.run_overlap(A, B, C, bufs=None, out=out, reduce_own=True, n_iter=n_iter, reps=1, warmup=0,
                    flags=occ.OCC_RUN_OVL, timeline=tl)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy().view(np.uint32),
                          C[-1].view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1).astype(np.uint32) << 16)
    g, c = timeline_intervals(tl, n_iter)
    assert schedule.dependency_violations(g, c) == []
