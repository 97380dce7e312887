"""Pins the CPU oracle to facts fixed outside it (runs on the CPU).

Each check is chosen so that a plausible slip in the oracle -- a transposed
operand, a dropped term, a wrong index, a reassociated sum, double rounding,
a wrong tie rule -- fails at least one of them:

* GEMM, binary64 sum (acc="f64"): exact rational brute force
  (fractions.Fraction) followed by an independent round-to-nearest-even
  written here; a float64 BLAS cross-check within one bfloat16 ulp.
* GEMM, binary32 accumulation in increasing k (acc="f32", the default):
  hand-derived order probes (tests/golden/gemm_f32acc_order.txt) whose
  result differs from the exact sum and from the reversed order; within
  K * 2^-24 * sum |a b| of the exact sum (plus the final rounding) on random
  operands.
* Both: integer-valued operands whose sums are exact, checked against
  numpy's int64 matmul and torch's float32 -> bfloat16 conversion; identity
  and all-ones closed forms; both B layouts; blocks are slices of the full
  result.
* bfloat16 rounding: a hand-derived table (tests/golden/bf16_rne.txt).
* Chunk sum: order probes whose left-fold result differs from any other
  order (tests/golden/chunk_sum_order.txt); all-ones -> nchunks; integer
  chunks -> exact integer sums; brute force with binary32 rounding after
  every addition (double rounding through binary64 is innocuous for a sum of
  two binary32 values because 53 >= 2*24 + 2).
* Permutation: hand-derived example (tests/golden/permute_small.txt),
  identity, inverse round trip, numpy fancy indexing, bijection check.
"""
import math
import os
import struct
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers
def f32_bits(x):
    return struct.unpack("<I", struct.pack("<f", x))[0]


def bits_f32(u):
    return struct.unpack("<f", struct.pack("<I", u))[0]


def bf16_value(h):
    """Exact rational value of a finite bfloat16 bit pattern."""
    h = int(h) & 0xFFFF
    s = -1 if h & 0x8000 else 1
    e = (h >> 7) & 0xFF
    m = h & 0x7F
    assert e != 0xFF
    if e == 0:
        return s * Fraction(m, 1 << 7) * Fraction(1, 1 << 126)
    return s * (1 + Fraction(m, 1 << 7)) * (Fraction(2) ** (e - 127))


def rne_bf16_exact(q):
    """Round a Fraction to bfloat16 (ties to even), by exhaustive neighbour search."""
    if q == 0:
        return 0x0000
    sign = 0x8000 if q < 0 else 0
    a = abs(q)
    # all non-negative finite patterns are ordered by value; bisect on them
    lo, hi = 0, 0x7F7F
    if a >= bf16_value(0x7F7F) + (Fraction(2) ** 127 * Fraction(1, 256)):
        return sign | 0x7F80
    while hi - lo > 1:
        mid = (lo + hi) // 2
        if bf16_value(mid) <= a:
            lo = mid
        else:
            hi = mid
    if bf16_value(hi) <= a:
        lo = hi
        hi = lo + 1
    dlo = a - bf16_value(lo)
    dhi = bf16_value(hi) - a if hi <= 0x7F7F else None
    if dhi is None or dlo < dhi:
        r = lo
    elif dhi < dlo:
        r = hi
    else:
        r = lo if lo % 2 == 0 else hi
    return sign | r


def to_bf16_bits_torch(x_f32):
    """Library conversion float32 -> bfloat16 (round to nearest even)."""
    t = torch.from_numpy(np.ascontiguousarray(x_f32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f64(h):
    return (np.asarray(h, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


def random_bf16(shape, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    return (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)


# ---------------------------------------------------------------- bfloat16 rounding
def _golden_rows(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([c.strip() for c in line.split("|")])
    return rows


@pytest.mark.parametrize("row", _golden_rows("bf16_rne.txt"), ids=lambda r: r[0])
def test_bf16_rounding_table(row):
    value = eval(row[0], {"float": float})  # fixture expressions are plain literals
    assert oracle.double_to_bf16(value) == int(row[1], 16)


def test_bf16_rounding_matches_exact_search():
    rng = np.random.default_rng(11)
    for _ in range(400):
        x = float(rng.standard_normal() * 2.0 ** rng.integers(-140, 120))
        assert oracle.double_to_bf16(x) == rne_bf16_exact(Fraction(x)), x


def test_bf16_roundtrip_all_finite_patterns():
    for h in range(0, 0x10000, 7):
        if (h >> 7) & 0xFF == 0xFF:
            continue
        assert oracle.double_to_bf16(oracle.bf16_to_double(h)) == h


# ---------------------------------------------------------------- GEMM
@pytest.mark.parametrize("M,N,K,seed", [(1, 1, 1, 0), (3, 4, 5, 1), (5, 3, 16, 2), (2, 7, 33, 3)])
def test_gemm_exact_rational(M, N, K, seed):
    A = random_bf16((M, K), seed)
    B = random_bf16((N, K), seed + 100)
    got = oracle.gemm_bf16(A, B, M, N, K, acc="f64")
    a = A.view(torch.int16).numpy().view(np.uint16)
    b = B.view(torch.int16).numpy().view(np.uint16)
    for m in range(M):
        for n in range(N):
            exact = sum(bf16_value(a[m, k]) * bf16_value(b[n, k]) for k in range(K))
            assert got[m, n] == rne_bf16_exact(exact), (m, n)


@pytest.mark.parametrize("row", _golden_rows("gemm_f32acc_order.txt"), ids=lambda r: r[0])
def test_gemm_accumulation_order_probes(row):
    a = [eval(v) for v in row[0].split(",")]
    b = [eval(v) for v in row[1].split(",")]
    K = len(a)
    A = torch.tensor([a], dtype=torch.float32).to(torch.bfloat16)
    B = torch.tensor([b], dtype=torch.float32).to(torch.bfloat16)      # N x K, N = 1
    assert A.float().tolist()[0] == a and B.float().tolist()[0] == b   # the values are bf16
    assert oracle.gemm_bf16(A, B, 1, 1, K, acc="f32")[0, 0] == int(row[2], 16)
    assert oracle.gemm_bf16(A, B, 1, 1, K, acc="f64")[0, 0] == int(row[3], 16)
    # the same with B stored K x N
    assert oracle.gemm_bf16(A, B.t().contiguous(), 1, 1, K, b_layout="kn")[0, 0] == int(row[2], 16)


@pytest.mark.parametrize("M,N,K,seed", [(16, 24, 512, 5), (9, 40, 2048, 6)])
def test_gemm_f32_accumulation_within_bound_of_exact(M, N, K, seed):
    A = random_bf16((M, K), seed)
    B = random_bf16((N, K), seed + 1)
    got = bf16_bits_to_f64(oracle.gemm_bf16(A, B, M, N, K, acc="f32"))
    a, b = A.double().numpy(), B.double().numpy()
    exact = a @ b.T                          # float64 BLAS: error far below the bound
    bound = K * 2.0 ** -24 * (np.abs(a) @ np.abs(b).T)
    half_ulp = np.maximum(np.abs(exact) + bound, 2.0 ** -126) * 2.0 ** -8
    assert np.all(np.abs(got - exact) <= bound + half_ulp)
    # and the two definitions agree on most outputs
    same = oracle.gemm_bf16(A, B, M, N, K, acc="f32") == oracle.gemm_bf16(A, B, M, N, K, acc="f64")
    assert same.mean() > 0.95


@pytest.mark.parametrize("M,N,K", [(37, 29, 512), (64, 8, 136), (7, 130, 256)])
def test_gemm_integer_operands_exact(M, N, K):
    rng = np.random.default_rng(M * N + K)
    ai = rng.integers(-2, 3, size=(M, K))
    bi = rng.integers(-2, 3, size=(N, K))
    A = torch.from_numpy(ai.astype(np.float32)).to(torch.bfloat16)
    B = torch.from_numpy(bi.astype(np.float32)).to(torch.bfloat16)
    exact = ai @ bi.T                               # int64 library matmul
    want = to_bf16_bits_torch(exact.astype(np.float32))  # |sum| < 2^24: float32 is exact
    assert np.array_equal(oracle.gemm_bf16(A, B, M, N, K, acc="f32"), want)
    assert np.array_equal(oracle.gemm_bf16(A, B, M, N, K, acc="f64"), want)


def test_gemm_identity_and_ones():
    A = random_bf16((24, 40), 5)
    eye = torch.eye(40).to(torch.bfloat16)
    got = oracle.gemm_bf16(A, eye, 24, 40, 40)
    assert np.array_equal(got, A.view(torch.int16).numpy().view(np.uint16))
    ones_a = torch.ones((3, 512), dtype=torch.bfloat16)
    ones_b = torch.ones((5, 512), dtype=torch.bfloat16)
    assert np.all(oracle.gemm_bf16(ones_a, ones_b, 3, 5, 512) == 0x4400)  # 512.0


def test_gemm_zero_k_is_zero():
    A = torch.empty((4, 0), dtype=torch.bfloat16)
    B = torch.empty((6, 0), dtype=torch.bfloat16)
    assert np.all(oracle.gemm_bf16(A, B, 4, 6, 0) == 0)


def test_gemm_layouts_agree_and_blas_within_one_ulp():
    M, N, K = 48, 80, 384
    A = random_bf16((M, K), 21)
    Bnk = random_bf16((N, K), 22)
    Bkn = Bnk.t().contiguous()
    c_nk = oracle.gemm_bf16(A, Bnk, M, N, K, b_layout="nk", acc="f64")
    c_kn = oracle.gemm_bf16(A, Bkn, M, N, K, b_layout="kn", acc="f64")
    assert np.array_equal(c_nk, c_kn)
    assert np.array_equal(oracle.gemm_bf16(A, Bnk, M, N, K, b_layout="nk"),
                          oracle.gemm_bf16(A, Bkn, M, N, K, b_layout="kn"))
    ref = A.double().numpy() @ Bnk.double().numpy().T    # float64 BLAS
    got = bf16_bits_to_f64(c_nk)
    ulp = np.maximum(np.abs(ref), 2.0 ** -126) * 2.0 ** -7
    assert np.all(np.abs(got - ref) <= ulp)
    # an operand transposed by mistake would be far off
    assert np.max(np.abs(got - ref)) < 0.05 * np.max(np.abs(ref))


def test_gemm_block_is_slice_of_full():
    M, N, K = 70, 90, 64
    A = random_bf16((M, K), 31)
    B = random_bf16((N, K), 32)
    full = oracle.gemm_bf16(A, B, M, N, K)
    blk = oracle.gemm_bf16(A, B, M, N, K, rows=(13, 61), cols=(40, 89))
    assert np.array_equal(blk, full[13:61, 40:89])


# ---------------------------------------------------------------- chunk sum
@pytest.mark.parametrize("row", _golden_rows("chunk_sum_order.txt"), ids=lambda r: r[0])
def test_chunk_sum_order_probes(row):
    vals = [eval(v) for v in row[0].split(",")]
    chunks = np.array([[v] for v in vals], dtype=np.float32)
    got = oracle.chunk_sum_f32(chunks)
    assert f32_bits(float(got[0])) == int(row[1], 16)


def test_chunk_sum_all_ones_and_identity():
    for n in (1, 2, 3, 8, 17):
        out = oracle.chunk_sum_f32(np.ones((n, 1000), dtype=np.float32))
        assert np.all(out == n)
    x = np.random.default_rng(3).standard_normal((1, 777)).astype(np.float32)
    assert np.array_equal(oracle.chunk_sum_f32(x).view(np.uint32), x[0].view(np.uint32))


def test_chunk_sum_integer_valued_exact():
    rng = np.random.default_rng(4)
    ci = rng.integers(-1024, 1025, size=(8, 5000))
    out = oracle.chunk_sum_f32(ci.astype(np.float32))
    assert np.array_equal(out, ci.sum(axis=0).astype(np.float32))


def test_chunk_sum_brute_force_binary32():
    rng = np.random.default_rng(5)
    c = (rng.random((6, 300)) * 2 - 1).astype(np.float32)
    c[:, :50] *= np.float32(2.0 ** 20)       # mixed magnitudes so rounding happens
    got = oracle.chunk_sum_f32(c)
    for j in range(c.shape[1]):
        acc = float(c[0, j])
        for i in range(1, c.shape[0]):
            acc = bits_f32(f32_bits(acc + float(c[i, j])))   # round to binary32 each add
        assert f32_bits(float(got[j])) == f32_bits(acc), j


# ------------------------------------------------ chunk sum with a bf16 own term
def _widen(u16):
    """bf16 bit patterns -> float32 by placing them in the high half (exact)."""
    return (np.asarray(u16, dtype=np.uint32) << 16).view(np.float32)


def test_chunk_sum_own_without_peers_is_the_widened_own_term():
    # every bf16 pattern, no peer chunks: out is the pattern widened, bit for
    # bit, and its value is the bf16 value (checked through the GEMM's own
    # bf16 -> double conversion for every non-NaN pattern)
    own = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = oracle.chunk_sum_own_f32(own, np.zeros((0, own.size), dtype=np.float32))
    assert np.array_equal(got.view(np.uint32), (own.astype(np.uint32) << 16))
    for h in range(0, 1 << 16, 97):
        v = oracle.bf16_to_double(h)
        if not math.isnan(v):
            assert float(got[h]) == v, hex(h)


def test_chunk_sum_own_order_own_first():
    # ((1 + 2^24) - 2^24) = 0 in binary32 (1 + 2^24 rounds to 2^24), while any
    # other grouping or own-last order gives 1: the own term comes first and
    # the fold is strictly left to right
    own = np.array([0x3F80], dtype=np.uint16)                      # 1.0
    peers = np.array([[2.0 ** 24], [-(2.0 ** 24)]], dtype=np.float32)
    assert oracle.chunk_sum_own_f32(own, peers)[0] == 0.0
    assert oracle.chunk_sum_f32(np.vstack([peers, [[1.0]]]).astype(np.float32))[0] == 1.0


def test_chunk_sum_own_integer_valued_exact_and_equal_to_widened_chunk_sum():
    rng = np.random.default_rng(6)
    own_i = rng.integers(-128, 129, size=4000)                     # exact in bf16
    own = (np.asarray(own_i, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(_widen(own), own_i.astype(np.float32))
    peers = rng.integers(-1024, 1025, size=(7, 4000))
    got = oracle.chunk_sum_own_f32(own, peers.astype(np.float32))
    assert np.array_equal(got, (own_i + peers.sum(axis=0)).astype(np.float32))
    # with rounding: the same as the plain chunk sum whose first chunk is the widened own term
    x = (rng.random((5, 999)) * 2 - 1).astype(np.float32) * np.float32(3.0e4)
    own2 = (x[0].view(np.uint32) >> 16).astype(np.uint16)
    ref = oracle.chunk_sum_f32(np.vstack([_widen(own2)[None, :], x[1:]]))
    assert np.array_equal(oracle.chunk_sum_own_f32(own2, x[1:]).view(np.uint32), ref.view(np.uint32))


def test_chunk_sum_own_special_values():
    own = np.array([0x7F80, 0xFF80, 0x7FC0, 0x0001, 0x8000], dtype=np.uint16)  # inf, -inf, nan, min subnormal, -0
    peers = np.zeros((1, 5), dtype=np.float32)
    got = oracle.chunk_sum_own_f32(own, peers)
    assert np.isposinf(got[0]) and np.isneginf(got[1]) and np.isnan(got[2])
    assert got[3] == np.float32(2.0 ** -133)
    assert got[4] == 0.0      # -0 + (+0) = +0 in round-to-nearest


# ---------------------------------------------------------------- permutation
def test_permute_golden():
    rows = {r[0]: r[1] for r in _golden_rows("permute_small.txt")}
    src = np.array([int(b, 16) for b in rows["src"].split()], dtype=np.uint8)
    perm = [int(p) for p in rows["perm"].split()]
    want = np.array([int(b, 16) for b in rows["dst"].split()], dtype=np.uint8)
    assert np.array_equal(oracle.permute_chunks(src, perm, 3), want)


def test_permute_identity_inverse_and_fancy_indexing():
    rng = np.random.default_rng(6)
    n, cb = 16, 96
    src = rng.integers(0, 256, size=n * cb, dtype=np.uint8)
    ident = list(range(n))
    assert np.array_equal(oracle.permute_chunks(src, ident, cb), src)
    p = rng.permutation(n)
    once = oracle.permute_chunks(src, p, cb)
    assert np.array_equal(once, src.reshape(n, cb)[p].reshape(-1))
    back = oracle.permute_chunks(once, np.argsort(p), cb)
    assert np.array_equal(back, src)


def test_permute_rejects_non_bijection():
    with pytest.raises(ValueError):
        oracle.permute_chunks(np.zeros(8, dtype=np.uint8), [0, 0, 1, 2], 2)


# ---------------------------------------------------------------- sanity of the helper itself
def test_exact_rounding_helper_matches_torch_on_float32():
    rng = np.random.default_rng(7)
    x = (rng.standard_normal(300) * 10).astype(np.float32)
    want = to_bf16_bits_torch(x)
    for v, w in zip(x, want):
        assert rne_bf16_exact(Fraction(float(v))) == int(w)
    assert math.isfinite(float(bf16_value(0x7F7F)))


def test_oracle_reports_its_thread_count():
    # bench.py's cpu_baseline states the threads the oracle ran on
    assert 1 <= oracle.num_threads() <= 4096
