"""Helpers shared by the GPU parity tests (comparison logic only)."""
import math

import numpy as np
import torch

DEV = "cuda:0"


def bf16_bits(t):
    """uint16 numpy array of a bfloat16 tensor's bit patterns (on the host)."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def bits_to_f64(h):
    return (np.asarray(h, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


def gemm_tolerance(std_a, std_b, K):
    """(rtol, atol) for bf16 outputs of an fp32-accumulated GEMM vs the oracle.

    rtol = 2e-2: bf16 inputs with fp32 accumulation; the two results differ
    by the fp32 summation error (about sqrt(K) * 2^-24 of the output's scale)
    plus at most one bf16 rounding step (2^-7 relative).  atol is 1/64 of the
    expected output magnitude std_a * std_b * sqrt(K), times rtol, so that
    outputs that cancel to near zero are judged on the output's scale; a wrong
    tile, index or operand produces errors of the order of that scale itself.
    """
    rtol = 2e-2
    atol = rtol * std_a * std_b * math.sqrt(max(K, 1)) / 64.0
    return rtol, atol


def assert_gemm_close(got_bits, ref_bits, std_a, std_b, K, what=""):
    """Element-wise |got - ref| <= rtol*|ref| + atol; returns the fraction of outputs not bit-identical."""
    got = bits_to_f64(got_bits)
    ref = bits_to_f64(ref_bits)
    rtol, atol = gemm_tolerance(std_a, std_b, K)
    both_nan = np.isnan(got) & np.isnan(ref)
    err = np.where(both_nan, 0.0, np.abs(got - ref))
    bad = ~(err <= rtol * np.abs(ref) + atol)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError("%s: %d of %d outputs outside tolerance, first at %s: got %s want %s"
                             % (what, int(bad.sum()), bad.size, idx.tolist(),
                                got[tuple(idx[0])], ref[tuple(idx[0])]))
    return float(np.mean(np.asarray(got_bits) != np.asarray(ref_bits)))


def sample_tiles(M, N, tile=64, count=32, seed=7):
    """`count` tile origins (m0, n0) on a `tile` grid, always including the four corners."""
    tm = max(1, math.ceil(M / tile))
    tn = max(1, math.ceil(N / tile))
    corners = {(0, 0), (0, tn - 1), (tm - 1, 0), (tm - 1, tn - 1)}
    rng = np.random.default_rng(seed)
    picks = list(corners)
    while len(picks) < min(count, tm * tn):
        p = (int(rng.integers(tm)), int(rng.integers(tn)))
        if p not in picks:
            picks.append(p)
    return [(a * tile, b * tile) for a, b in picks]
