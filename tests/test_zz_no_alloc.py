"""occ_overlap_enqueue_noalloc against occ_overlap_enqueue: the same kernels
with the counters in the library's static device array instead of a caller
workspace.  Two calls in a row, the second with a smaller input (fewer
iterations, a smaller GEMM and a shorter collective); outputs bit-identical
to the workspace entry point's, no timeout reported."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_09200_amd import binding as occ
from paper_2606_09200_amd import inputs
from gpu_common import DEV, assert_gemm_close, bf16_bits

pytestmark = pytest.mark.gpu


def _case(M, N, K, n_iter, kind, seed):
    A, Bt = inputs.gemm_operands(M, N, K, seed=seed, device=DEV)
    B = Bt.t().contiguous()
    if kind == "own":
        C = torch.full((n_iter, M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
        comm = dict(bufs=inputs.reduce_chunks(2, M * N, seed=seed + 1, device=DEV),
                    out=torch.full((M * N,), float("nan"), device=DEV), reduce_own=True)
        outk = "out"
    elif kind == "reduce":
        C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
        length = M * N * 3 + 5                     # ragged: a scalar tail kernel too
        comm = dict(bufs=inputs.reduce_chunks(4, length, seed=seed + 1, device=DEV),
                    out=torch.full((length,), float("nan"), device=DEV))
        outk = "out"
    else:
        C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
        src = inputs.permute_payload(8, M * 64, seed=seed + 1, device=DEV)
        comm = dict(src=src, dst=torch.zeros_like(src), perm=inputs.chunk_permutation(8, seed=seed),
                    chunk_bytes=M * 64)
        outk = "dst"
    return A, B, C, comm, outk


@pytest.mark.parametrize("kind", ["reduce", "permute", "own"])
def test_enqueue_noalloc_matches_workspace_entry_point(kind):
    s1 = torch.cuda.Stream()
    for M, N, K, n_iter in ((1024, 768, 512, 8), (264, 136, 200, 3)):   # the second call smaller
        A, B, C, comm, outk = _case(M, N, K, n_iter, kind, seed=M)
        ws = torch.zeros(occ.occ_overlap_workspace_bytes(n_iter) // 4, dtype=torch.int32, device=DEV)
        err_ws = torch.zeros(1, dtype=torch.int32, device=DEV)
        torch.cuda.synchronize()
        occ.occ_overlap_enqueue(A, B, C, workspace=ws, comm_stream=s1, err=err_ws, n_iter=n_iter, **comm)
        torch.cuda.synchronize()
        C_ws, out_ws = C.clone(), comm[outk].clone()
        C.fill_(float("nan"))
        comm[outk].fill_(0)
        err = torch.zeros(1, dtype=torch.int32, device=DEV)
        torch.cuda.synchronize()
        occ.occ_overlap_enqueue_noalloc(A, B, C, comm_stream=s1, err=err, n_iter=n_iter, **comm)
        torch.cuda.synchronize()
        assert int(err.item()) == 0 and int(err_ws.item()) == 0
        assert torch.equal(C.view(torch.int16), C_ws.view(torch.int16)), (M, N, K)
        assert torch.equal(comm[outk].view(torch.uint8), out_ws.view(torch.uint8)), (M, N, K)
        # and the outputs are the oracle's
        Cl = C[-1] if kind == "own" else C
        ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), M, N, K, b_layout="kn")
        assert_gemm_close(bf16_bits(Cl), ref, 1.0, 1.0, K, "noalloc C")
        if kind == "reduce":
            want = oracle.chunk_sum_f32(comm["bufs"].cpu().numpy())
            assert np.array_equal(comm["out"].cpu().numpy().view(np.uint32), want.view(np.uint32))
        elif kind == "own":
            want = oracle.chunk_sum_own_f32(C[-1].cpu(), comm["bufs"].cpu().numpy())
            assert np.array_equal(comm["out"].cpu().numpy().view(np.uint32), want.view(np.uint32))
        else:
            want = oracle.permute_chunks(comm["src"].cpu().numpy(), comm["perm"].numpy(), comm["chunk_bytes"])
            assert np.array_equal(comm["dst"].cpu().numpy(), want)


def test_enqueue_noalloc_back_to_back_without_host_sync():
    """Four schedules in a row on the library's array, each one's GEMM stream
    ordered after the previous one's collectives by a stream event only (no
    host synchronisation): every output is the oracle's and no wait runs
    out, so each schedule left the array at zero for the next."""
    M, N, K, n_iter = 264, 136, 200, 5
    A, B, _, _, _ = _case(M, N, K, n_iter, "reduce", seed=7)
    rounds = 4
    Cs = [torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16) for _ in range(rounds)]
    chunks = [inputs.reduce_chunks(3, 70001, seed=20 + r, device=DEV) for r in range(rounds)]
    outs = [torch.full((70001,), float("nan"), device=DEV) for _ in range(rounds)]
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    s0 = torch.cuda.current_stream()
    s1 = torch.cuda.Stream()
    torch.cuda.synchronize()
    for r in range(rounds):
        occ.occ_overlap_enqueue_noalloc(A, B, Cs[r], comm_stream=s1, err=err, n_iter=n_iter, bufs=chunks[r],
                                        out=outs[r])
        done = torch.cuda.Event()
        done.record(s1)
        s0.wait_event(done)
    torch.cuda.synchronize()
    assert int(err.item()) == 0
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), M, N, K, b_layout="kn")
    for r in range(rounds):
        assert_gemm_close(bf16_bits(Cs[r]), ref, 1.0, 1.0, K, "noalloc C, round %d" % r)
        want = oracle.chunk_sum_f32(chunks[r].cpu().numpy())
        assert np.array_equal(outs[r].cpu().numpy().view(np.uint32), want.view(np.uint32)), r


def test_enqueue_noalloc_rejects_more_iterations_than_its_array():
    A, B, C, comm, _ = _case(264, 136, 200, 1, "reduce", seed=1)
    s1 = torch.cuda.Stream()
    with pytest.raises(occ.OccError) as e:
        occ.occ_overlap_enqueue_noalloc(A, B, C, comm_stream=s1, n_iter=occ.NOALLOC_MAX_ITER + 1, **comm)
    assert e.value.status == occ.OCC_EINVAL
