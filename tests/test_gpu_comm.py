"""Parity of the communication-side kernels (through the C ABI) with the oracle:
bit-exact for the fixed-order chunk sum and for the chunk permutation."""
import os
import struct

import numpy as np
import pytest
import torch

import oracle
from paper_2606_09200_amd import binding as occ
from paper_2606_09200_amd import inputs
from gpu_common import DEV

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def gpu_reduce(chunks_host, offset=0, wgs=0, priority=0):
    """Run share_reduce on copies of the rows of chunks_host, optionally
    placed `offset` floats into their buffers (to exercise misalignment)."""
    n, length = chunks_host.shape
    store = torch.zeros((n, length + offset + 4), dtype=torch.float32, device=DEV)
    store[:, offset:offset + length] = torch.from_numpy(np.ascontiguousarray(chunks_host)).to(DEV)
    bufs = [store[i, offset:offset + length] for i in range(n)]
    out_store = torch.full((length + offset + 4,), float("nan"), dtype=torch.float32, device=DEV)
    out = out_store[offset:offset + length]
    occ.share_reduce(bufs, out, wgs=wgs, priority=priority)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def u32(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def own_bits(length, seed):
    """bf16 bit patterns of N(0,1) samples (no signalling NaNs)."""
    g = torch.Generator().manual_seed(seed)
    return torch.randn(length, generator=g).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def gpu_reduce_own(own_host, peers_host, own_offset=0, offset=0, wgs=0, priority=0):
    """share_reduce_own on device copies; `own_offset` bf16 elements and
    `offset` floats into their buffers (to exercise misalignment)."""
    n, length = peers_host.shape
    ostore = torch.zeros(length + own_offset + 8, dtype=torch.int16, device=DEV)
    ostore[own_offset:own_offset + length] = torch.from_numpy(own_host.view(np.int16)).to(DEV)
    own = ostore[own_offset:own_offset + length].view(torch.bfloat16)
    store = torch.zeros((max(n, 1), length + offset + 4), dtype=torch.float32, device=DEV)
    if n:
        store[:n, offset:offset + length] = torch.from_numpy(np.ascontiguousarray(peers_host)).to(DEV)
    peers = [store[i, offset:offset + length] for i in range(n)]
    out_store = torch.full((length + offset + 4,), float("nan"), dtype=torch.float32, device=DEV)
    out = out_store[offset:offset + length]
    occ.share_reduce_own(own, peers, out, wgs=wgs, priority=priority)
    torch.cuda.synchronize()
    return out.cpu().numpy()


@pytest.mark.parametrize("n", [0, 1, 3, 5, 7, 15, 20, 63])
@pytest.mark.parametrize("length", [1, 3, 4, 1000, 65539])
def test_reduce_own_bit_exact(n, length):
    own = own_bits(length, seed=n + 7 * length)
    peers = inputs.reduce_chunks(n, length, seed=n * 1000 + length).numpy() if n else np.zeros((0, length), np.float32)
    got = gpu_reduce_own(own, peers)
    assert np.array_equal(u32(got), u32(oracle.chunk_sum_own_f32(own, peers)))


@pytest.mark.parametrize("own_offset,offset", [(1, 0), (2, 0), (3, 1), (0, 2), (4, 0)])
def test_reduce_own_misaligned_bit_exact(own_offset, offset):
    own = own_bits(4099, seed=own_offset)
    peers = inputs.reduce_chunks(7, 4099, seed=11).numpy()
    got = gpu_reduce_own(own, peers, own_offset=own_offset, offset=offset)
    assert np.array_equal(u32(got), u32(oracle.chunk_sum_own_f32(own, peers)))


def test_reduce_own_order_and_specials():
    # ((1 + 2^24) - 2^24) = 0: own first, strict left fold; special bf16 values widen exactly
    own = np.array([0x3F80, 0x7F80, 0xFF80, 0x0001, 0x8000, 0x3F80, 0x4000, 0xC000], dtype=np.uint16)
    peers = np.zeros((2, 8), dtype=np.float32)
    peers[:, 0] = [2.0 ** 24, -(2.0 ** 24)]
    got = gpu_reduce_own(own, peers)
    ref = oracle.chunk_sum_own_f32(own, peers)
    assert got[0] == 0.0 and np.array_equal(u32(got), u32(ref))
    got0 = gpu_reduce_own(own, np.zeros((0, 8), dtype=np.float32))
    assert np.array_equal(u32(got0), own.astype(np.uint32) << 16)


@pytest.mark.parametrize("wgs,priority", [(1, 0), (3, 3), (1000, 1)])
def test_reduce_own_knobs_do_not_change_bits(wgs, priority):
    own = own_bits(70001, seed=5)
    peers = inputs.reduce_chunks(3, 70001, seed=6).numpy()
    assert np.array_equal(u32(gpu_reduce_own(own, peers, wgs=wgs, priority=priority)),
                          u32(oracle.chunk_sum_own_f32(own, peers)))


def test_reduce_own_workload_size_bit_exact():
    # the cb_own share: the 8192 x 8192 GEMM output and 7 fp32 peer chunks
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS["cb_own"]
    length = w.M * w.N
    own = torch.randn(length, device=DEV).to(torch.bfloat16)
    peers = inputs.reduce_chunks(w.nchunks, length, seed=1, device=DEV)
    out = torch.empty(length, device=DEV)
    occ.share_reduce_own(own, peers, out)
    torch.cuda.synchronize()
    ref = oracle.chunk_sum_own_f32(own.cpu(), peers.cpu().numpy())
    assert np.array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 8, 9, 16, 17, 64])
@pytest.mark.parametrize("length", [1, 3, 4, 1000, 65539])
def test_reduce_bit_exact(n, length):
    c = inputs.reduce_chunks(n, length, seed=n * 1000 + length).numpy()
    assert np.array_equal(u32(gpu_reduce(c)), u32(oracle.chunk_sum_f32(c)))


@pytest.mark.parametrize("offset", [1, 2, 3])
def test_reduce_misaligned_bit_exact(offset):
    c = inputs.reduce_chunks(8, 4099, seed=offset).numpy()
    assert np.array_equal(u32(gpu_reduce(c, offset=offset)), u32(oracle.chunk_sum_f32(c)))


def test_reduce_order_probes():
    with open(os.path.join(GOLDEN, "chunk_sum_order.txt")) as f:
        rows = [l.split("|") for l in f if l.strip() and not l.startswith("#")]
    for row in rows:
        vals = [eval(v) for v in row[0].split(",")]
        # 4100 copies so that both the vector body and the scalar tail see the probe
        c = np.repeat(np.array(vals, dtype=np.float32)[:, None], 4101, axis=1)
        got = u32(gpu_reduce(c))
        assert np.all(got == int(row[1], 16)), row[0]


def test_reduce_mixed_magnitudes_and_subnormals():
    rng = np.random.default_rng(9)
    c = (rng.standard_normal((8, 20000)) * np.float32(2.0) ** rng.integers(-140, 100, size=(8, 20000))).astype(np.float32)
    c[3, ::7] = np.float32(1e-45)           # smallest subnormal
    c[5, ::11] = -c[0, ::11]                # exact cancellations
    assert np.array_equal(u32(gpu_reduce(c)), u32(oracle.chunk_sum_f32(c)))


def test_reduce_infinities_overflow_and_nan():
    # IEEE binary32 in the fixed order: overflow to +-inf, inf + finite, and
    # NaN from inf + -inf or a NaN term (NaN payloads are the hardware's, so
    # NaN positions are compared as a set and every other result bit-exact)
    rng = np.random.default_rng(21)
    L = 4099
    c = rng.standard_normal((8, L)).astype(np.float32)
    big = np.finfo(np.float32).max
    c[0, ::23] = big
    c[1, ::23] = big                        # overflow to +inf after the second term
    c[6, ::29] = -big
    c[2, ::13] = np.inf
    c[4, ::17] = -np.inf                    # inf + -inf = NaN every 221st element
    c[7, ::19] = np.nan
    c[3, 5] = np.float32(2.0 ** 127)        # one term that stays finite
    got = gpu_reduce(c)
    ref = oracle.chunk_sum_f32(c)
    nan_got, nan_ref = np.isnan(got), np.isnan(ref)
    assert nan_ref.any() and np.isinf(ref).any()
    assert np.array_equal(nan_got, nan_ref)
    assert np.array_equal(u32(got[~nan_ref]), u32(ref[~nan_ref]))


def test_reduce_all_ones_and_integers():
    assert np.all(gpu_reduce(np.ones((8, 5000), dtype=np.float32)) == 8.0)
    ci = np.random.default_rng(4).integers(-1024, 1025, size=(8, 5000))
    assert np.array_equal(gpu_reduce(ci.astype(np.float32)), ci.sum(axis=0).astype(np.float32))


@pytest.mark.parametrize("wgs,priority", [(1, 0), (3, 3), (1000, 1), (0, 2)])
def test_reduce_knobs_do_not_change_bits(wgs, priority):
    c = inputs.reduce_chunks(8, 300001, seed=2).numpy()
    assert np.array_equal(u32(gpu_reduce(c, wgs=wgs, priority=priority)), u32(oracle.chunk_sum_f32(c)))


def test_reduce_empty_is_noop():
    out = torch.full((4,), 7.0, device=DEV)
    bufs = [torch.zeros(4, device=DEV)[:0]]
    occ.lib().share_reduce((occ.ctypes.c_void_p * 1)(bufs[0].data_ptr()), 1, 0, occ._ptr(out), occ._stream(None))
    torch.cuda.synchronize()
    assert torch.all(out == 7.0)


# paper_cb_ar: Table 1's 896 MiB allreduce share, 4 chunks of 224 MiB
@pytest.mark.parametrize("name", ["tiny", "mb", "cb", "paper_cb_ar"])
def test_reduce_workload_sizes_bit_exact(name):
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS[name]
    chunks = inputs.reduce_chunks(w.nchunks, w.length, seed=1, device=DEV)
    out = torch.empty(w.length, device=DEV)
    occ.share_reduce(chunks, out)
    torch.cuda.synchronize()
    ref = oracle.chunk_sum_f32(chunks.cpu().numpy())
    assert np.array_equal(u32(out.cpu().numpy()), u32(ref))


# ----------------------------------------------------------------- permutation
def gpu_permute(src_host, perm, chunk_bytes, byte_offset=0, wgs=0, priority=0):
    total = src_host.size
    s = torch.zeros(total + 64, dtype=torch.uint8, device=DEV)
    s[byte_offset:byte_offset + total] = torch.from_numpy(src_host).to(DEV)
    d = torch.zeros(total + 64, dtype=torch.uint8, device=DEV)
    occ.share_permute(s[byte_offset:byte_offset + total], d[byte_offset:byte_offset + total], perm,
                      chunk_bytes, wgs=wgs, priority=priority)
    torch.cuda.synchronize()
    return d[byte_offset:byte_offset + total].cpu().numpy()


# 16 * (3 * 1024 + 517): three full unrolled trips of a 128-lane workgroup
# and a ragged tail; 16 * (2 * 16384 + 123): one chunk split into three work
# items of unequal length.
@pytest.mark.parametrize("n,cb", [(1, 16), (4, 4096), (64, 65536), (7, 1040), (512, 48), (3, 1001), (5, 17),
                                  (3, 16 * (3 * 1024 + 517)), (2, 16 * (2 * 16384 + 123))])
def test_permute_bit_exact(n, cb):
    src = inputs.permute_payload(n, cb, seed=n + cb).numpy()
    perm = inputs.chunk_permutation(n, seed=n)
    want = oracle.permute_chunks(src, perm.numpy(), cb)
    assert np.array_equal(gpu_permute(src, perm, cb), want)


@pytest.mark.parametrize("offset", [1, 8])
def test_permute_misaligned_bit_exact(offset):
    src = inputs.permute_payload(6, 4096, seed=offset).numpy()
    perm = inputs.chunk_permutation(6, seed=offset)
    want = oracle.permute_chunks(src, perm.numpy(), 4096)
    assert np.array_equal(gpu_permute(src, perm, 4096, byte_offset=offset), want)


def test_permute_identity_and_round_trip():
    src = inputs.permute_payload(32, 8192, seed=5).numpy()
    ident = list(range(32))
    assert np.array_equal(gpu_permute(src, ident, 8192), src)
    p = inputs.chunk_permutation(32, seed=6).numpy()
    once = gpu_permute(src, p, 8192)
    assert np.array_equal(gpu_permute(once, np.argsort(p), 8192), src)


@pytest.mark.parametrize("wgs,priority", [(1, 3), (7, 0), (4096, 2)])
def test_permute_knobs_do_not_change_bits(wgs, priority):
    src = inputs.permute_payload(16, 1 << 16, seed=8).numpy()
    perm = inputs.chunk_permutation(16, seed=8)
    want = oracle.permute_chunks(src, perm.numpy(), 1 << 16)
    assert np.array_equal(gpu_permute(src, perm, 1 << 16, wgs=wgs, priority=priority), want)


# paper_cb_a2a: Table 1's 896 MiB alltoall share, 4 chunks of 224 MiB
@pytest.mark.parametrize("name", ["a2a", "paper_cb_a2a"])
def test_permute_workload_size_bit_exact(name):
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS[name]
    src = inputs.permute_payload(w.nchunks, w.chunk_bytes, seed=2, device=DEV)
    perm = inputs.chunk_permutation(w.nchunks, seed=3)
    dst = torch.empty_like(src)
    occ.share_permute(src, dst, perm, w.chunk_bytes)
    torch.cuda.synchronize()
    want = oracle.permute_chunks(src.cpu().numpy(), perm.numpy(), w.chunk_bytes)
    assert np.array_equal(dst.cpu().numpy(), want)


# ------------------------------------------------------------ beyond 4 GiB
def _sample_positions(n, seed, around=()):
    rng = np.random.default_rng(seed)
    idx = set(rng.integers(0, n, 4096).tolist())
    idx.update(range(0, 64))
    idx.update(range(max(0, n - 64), n))
    for a in around:
        idx.update(range(max(0, a - 64), min(n, a + 64)))
    return torch.tensor(sorted(idx), dtype=torch.int64)


def test_reduce_chunks_beyond_4gib_sampled():
    """Chunks of 2^30 + 1027 floats (just over 4 GiB each): the kernel's byte
    offsets no longer fit in 32 bits, so the 64-bit addressing path runs; the
    scalar tail covers the last 3 elements.  Checked at sampled positions,
    including both sides of the 2^32-byte boundary, against the oracle."""
    n = (1 << 30) + 1027
    g = torch.Generator(device=DEV)
    g.manual_seed(11)
    chunks = torch.rand((2, n), generator=g, device=DEV, dtype=torch.float32)
    out = torch.full((n,), float("nan"), device=DEV)
    occ.share_reduce(chunks, out)
    torch.cuda.synchronize()
    pos = _sample_positions(n, 1, around=((1 << 30), (1 << 28)))
    p = pos.to(DEV)
    got = out[p].cpu().numpy()
    want = oracle.chunk_sum_f32(np.ascontiguousarray(chunks[:, p].cpu().numpy()))
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
    del chunks, out
    torch.cuda.empty_cache()


def test_permute_chunks_beyond_4gib_sampled():
    """Two chunks of 4 GiB + 4096 B, swapped: 64-bit offsets inside a chunk."""
    cb = (1 << 32) + 4096
    src = torch.empty(2 * cb, dtype=torch.uint8, device=DEV)
    g = torch.Generator(device=DEV)
    g.manual_seed(12)
    src.view(torch.int32).random_(generator=g)
    dst = torch.zeros_like(src)
    perm = torch.tensor([1, 0], dtype=torch.int32)
    occ.share_permute(src, dst, perm, cb)
    torch.cuda.synchronize()
    pos = _sample_positions(cb, 2, around=((1 << 32),))
    p = pos.to(DEV)
    for i in range(2):
        j = int(perm[i])
        assert torch.equal(dst[i * cb + p], src[j * cb + p]), i
    del src, dst
    torch.cuda.empty_cache()
