"""Seeded synthetic inputs shared by the HIP path, the tests and the benchmark.

This module only draws random numbers; it performs none of the method's
arithmetic.  The paper trains on no public dataset for this path: its GEMM
shapes come from LLaMA training at sequence length 8192 (Section 4.1) and
its collectives carry synthetic payloads, so every operand here is drawn from
a seeded generator with the distribution the workload names:

* GEMM operands: normal, given standard deviation, stored as bfloat16 (the
  float32 draw is rounded to nearest-even by torch's conversion);
* allreduce chunks: float32 uniform on [-1, 1), i.e. 2*U[0,1) - 1;
* alltoall payload: uniformly random 16-bit patterns (any bfloat16 bits,
  NaNs included) and a uniformly random permutation of the chunk indices.

With ``device="cpu"`` the draws come from torch's CPU generator and are
reproducible across machines; with a GPU device they come from torch's GPU
generator (still seeded and deterministic for one torch build), which is
faster for the largest workloads.
"""
import torch


def _gen(seed, device):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def gemm_operands(M, N, K, seed=0, std_a=1.0, std_b=1.0, seed_b=None, device="cpu"):
    """A (M x K) and B (N x K, a linear layer's weight layout), both bfloat16.

    A is drawn first, then B, from one generator seeded with ``seed``;
    ``seed_b`` gives B a generator of its own.
    """
    g = _gen(seed, device)
    A = torch.randn((M, K), generator=g, device=device, dtype=torch.float32)
    if std_a != 1.0:
        A.mul_(std_a)
    gb = g if seed_b is None else _gen(seed_b, device)
    B = torch.randn((N, K), generator=gb, device=device, dtype=torch.float32)
    if std_b != 1.0:
        B.mul_(std_b)
    return A.to(torch.bfloat16), B.to(torch.bfloat16)


def reduce_chunks(nchunks, length, seed=1, device="cpu"):
    """float32 (nchunks x length), uniform on [-1, 1)."""
    g = _gen(seed, device)
    x = torch.rand((nchunks, length), generator=g, device=device, dtype=torch.float32)
    return x.mul_(2.0).sub_(1.0)


def permute_payload(nchunks, chunk_bytes, seed=2, device="cpu"):
    """Random bytes (nchunks * chunk_bytes,), drawn as uniformly random 16-bit words."""
    if chunk_bytes % 2:
        g = _gen(seed, device)
        return torch.randint(0, 256, (nchunks * chunk_bytes,), generator=g, device=device,
                             dtype=torch.uint8)
    g = _gen(seed, device)
    w = torch.randint(-32768, 32768, (nchunks * chunk_bytes // 2,), generator=g,
                      device=device, dtype=torch.int16)
    return w.view(torch.uint8)


def chunk_permutation(nchunks, seed=3):
    """A uniformly random permutation of range(nchunks), int32 on the host."""
    g = _gen(seed, "cpu")
    return torch.randperm(nchunks, generator=g).to(torch.int32)
