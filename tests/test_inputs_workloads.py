"""The seeded input generators and the workload table (host only).

Inputs: deterministic per seed, the stated distributions (normal with the
given standard deviation, uniform on [-1, 1), 16-bit random patterns, a
bijective permutation) and independence of the two GEMM operands when B has
a seed of its own.  Workloads: the shapes and byte/flop counts the rooflines
use, written out from their definitions.
"""
import numpy as np
import pytest
import torch

from paper_2606_09200_amd import inputs
from paper_2606_09200_amd.workloads import BLOCK_COUNTS, WORKLOADS, MIB


def test_gemm_operands_seeded_and_distributed():
    A1, B1 = inputs.gemm_operands(256, 192, 512, seed=7)
    A2, B2 = inputs.gemm_operands(256, 192, 512, seed=7)
    assert A1.dtype == B1.dtype == torch.bfloat16
    assert A1.shape == (256, 512) and B1.shape == (192, 512)
    assert torch.equal(A1.view(torch.int16), A2.view(torch.int16))
    assert torch.equal(B1.view(torch.int16), B2.view(torch.int16))
    A3, _ = inputs.gemm_operands(256, 192, 512, seed=8)
    assert not torch.equal(A1.view(torch.int16), A3.view(torch.int16))
    a = A1.float().numpy()
    assert abs(a.mean()) < 0.02 and abs(a.std() - 1.0) < 0.02


def test_gemm_operand_std_and_own_seed_for_b():
    _, B = inputs.gemm_operands(4, 4096, 64, seed=0, std_b=0.02, seed_b=4)
    b = B.float().numpy()
    assert abs(b.std() - 0.02) < 0.001
    # B drawn from its own generator does not depend on A's shape or seed
    _, B2 = inputs.gemm_operands(9, 4096, 64, seed=5, std_b=0.02, seed_b=4)
    assert torch.equal(B.view(torch.int16), B2.view(torch.int16))


def test_reduce_chunks_uniform_on_minus_one_one():
    x = inputs.reduce_chunks(4, 1 << 16, seed=1)
    assert x.dtype == torch.float32 and x.shape == (4, 1 << 16)
    v = x.numpy()
    assert v.min() >= -1.0 and v.max() < 1.0
    assert abs(v.mean()) < 0.01 and abs(v.var() - 1.0 / 3.0) < 0.01
    assert torch.equal(x, inputs.reduce_chunks(4, 1 << 16, seed=1))


@pytest.mark.parametrize("chunk_bytes", [1 << 12, 4097])
def test_permute_payload_bytes(chunk_bytes):
    p = inputs.permute_payload(8, chunk_bytes, seed=2)
    assert p.dtype == torch.uint8 and p.numel() == 8 * chunk_bytes
    counts = np.bincount(p.numpy(), minlength=256)
    assert counts.min() > 0                      # every byte value occurs
    assert torch.equal(p, inputs.permute_payload(8, chunk_bytes, seed=2))


@pytest.mark.parametrize("n", [1, 2, 64, 512])
def test_chunk_permutation_is_a_seeded_bijection(n):
    p = inputs.chunk_permutation(n, seed=3)
    assert p.dtype == torch.int32
    assert sorted(p.tolist()) == list(range(n))
    assert torch.equal(p, inputs.chunk_permutation(n, seed=3))


def test_workload_table():
    w = WORKLOADS
    assert (w["cb"].M, w["cb"].N, w["cb"].K) == (8192, 8192, 8192)
    assert (w["mb"].M, w["mb"].N, w["mb"].K) == (16, 28672, 8192) and w["mb"].std_b == 0.02
    assert (w["a2a"].M, w["a2a"].N, w["a2a"].K) == (16384, 14336, 4096)
    assert w["a2a"].comm == "permute" and w["a2a"].nchunks == 64 and w["a2a"].chunk_bytes == 4 * MIB
    assert w["sweep"].pads == tuple(k << 10 for k in (0, 16, 32, 64, 96, 128))
    for name in ("paper_cb_ar", "paper_mb_ar", "paper_cb_a2a", "paper_mb_a2a"):
        x = w[name]
        share = x.nchunks * (x.length * 4 if x.comm == "reduce" else x.chunk_bytes)
        assert share == 896 * MIB, name
    assert BLOCK_COUNTS == (8, 16, 32, 64, 128)
    for x in w.values():
        assert x.gemm_flops == 2.0 * x.M * x.N * x.K
        assert x.gemm_bytes == 2.0 * (x.M * x.K + x.N * x.K + x.M * x.N)
        if x.comm == "reduce":
            assert x.comm_bytes == 4.0 * x.length * (x.nchunks + 1)
        elif x.comm == "reduce_own":
            assert x.length == x.M * x.N                  # the collective consumes C_i
            assert x.comm_bytes == 2.0 * x.length + 4.0 * x.length * (x.nchunks + 1)
        else:
            assert x.comm_bytes == 2.0 * x.nchunks * x.chunk_bytes
    assert w["cb_own"].comm == "reduce_own" and w["cb_own"].nchunks == 7
