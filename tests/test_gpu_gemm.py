"""GEMM parity: the HIP kernels (through the C ABI) against the CPU oracle.

occ_gemm is the contract C = A * B with B stored K x N; occ_gemm_bt is the
linear-layer form C = A * B^T with B stored N x K.  Both are checked against
the oracle's plain definition (exact products summed, one rounding to bf16)
at the tolerance derived in gpu_common.gemm_tolerance, and bit-exactly where
the sums are exact in fp32 (small-integer operands)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_09200_amd import binding as occ
from paper_2606_09200_amd import inputs
from gpu_common import DEV, assert_gemm_close, bf16_bits, sample_tiles

pytestmark = pytest.mark.gpu

KN_TILED = [32, 35, 36, 37, 38, 39]       # occ_gemm_ex, M > 16
KN_SKINNY = [33]                          # occ_gemm_ex, M <= 16
NK_TILED = [6, 7, 9, 14, 16, 25]          # occ_gemm_bt_ex, M > 16
NK_SKINNY = [21]                          # occ_gemm_bt_ex, M <= 16, any K
LDSB = 34                                 # occ_gemm_bt_ex, M <= 16, K % 1024 == 0, K <= 8192
OPT1_KN, OPT2_KN = 36, 37                 # the paper's Table 1 tiles, B K x N


def run_gemm(A, B, lds_bytes=0, variant=0, grid_cap=0):
    """occ_gemm(_ex) on host operands: A M x K, B K x N; returns C's bits."""
    M, K = A.shape
    N = B.shape[1]
    Ad, Bd = A.to(DEV), B.to(DEV)
    C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm_ex(Ad, Bd, C, lds_bytes=lds_bytes, variant=variant, grid_cap=grid_cap)
    torch.cuda.synchronize()
    return bf16_bits(C)


def run_gemm_bt(A, Bt, lds_bytes=0, variant=0, grid_cap=0):
    """occ_gemm_bt(_ex) on host operands: A M x K, Bt N x K; returns C's bits."""
    M, K = A.shape
    N = Bt.shape[0]
    Ad, Bd = A.to(DEV), Bt.to(DEV)
    C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm_bt_ex(Ad, Bd, C, lds_bytes=lds_bytes, variant=variant, grid_cap=grid_cap)
    torch.cuda.synchronize()
    return bf16_bits(C)


def operands(M, N, K, seed):
    """N(0,1) operands: A (M x K) and B stored K x N, with the same B stored N x K."""
    A, Bt = inputs.gemm_operands(M, N, K, seed=seed)
    return A, Bt.t().contiguous(), Bt


def int_operands(M, N, K, seed):
    """Entries in {-2..2}: every fp32 partial sum is exact, in any order."""
    g = torch.Generator().manual_seed(seed)
    A = torch.randint(-2, 3, (M, K), generator=g).to(torch.bfloat16)
    Bt = torch.randint(-2, 3, (N, K), generator=g).to(torch.bfloat16)
    return A, Bt.t().contiguous(), Bt


# ------------------------------------------------------------ occ_gemm (K x N)
@pytest.mark.parametrize("M,N,K", [(512, 512, 512), (300, 264, 136), (1, 8, 8), (17, 40, 64),
                                   (257, 136, 520), (64, 64, 32), (520, 1000, 1032), (16, 256, 4096),
                                   (600, 776, 200), (5, 80, 256), (7, 336, 6144), (2100, 2056, 264)])
def test_gemm_auto_full_parity(M, N, K):
    A, B, _ = operands(M, N, K, seed=4)
    got = run_gemm(A, B)
    ref = oracle.gemm_bf16(A, B, M, N, K, b_layout="kn")
    frac = assert_gemm_close(got, ref, 1.0, 1.0, K, "auto %dx%dx%d" % (M, N, K))
    assert frac < 0.05


@pytest.mark.parametrize("variant", KN_TILED + KN_SKINNY)
def test_gemm_every_variant_ragged(variant):
    # partial tiles in M and N, K not a multiple of the k-step
    M = 13 if variant in KN_SKINNY else 300
    N, K = 264, 200
    A, B, _ = operands(M, N, K, seed=variant)
    got = run_gemm(A, B, variant=variant)
    ref = oracle.gemm_bf16(A, B, M, N, K, b_layout="kn")
    assert_gemm_close(got, ref, 1.0, 1.0, K, "variant %d" % variant)


@pytest.mark.parametrize("variant", KN_TILED + KN_SKINNY)
def test_gemm_integer_operands_bit_exact(variant):
    M = 13 if variant in KN_SKINNY else 197
    A, B, _ = int_operands(M, 152, 520, seed=variant)
    got = run_gemm(A, B, variant=variant)
    assert np.array_equal(got, oracle.gemm_bf16(A, B, M, 152, 520, b_layout="kn"))


def _bf16_isnan(bits):
    return ((bits & 0x7F80) == 0x7F80) & ((bits & 0x007F) != 0)


@pytest.mark.parametrize("layout,variant", [("kn", v) for v in [0] + KN_TILED + KN_SKINNY] +
                         [("nk", v) for v in [0] + NK_TILED + NK_SKINNY + [LDSB]])
def test_gemm_infinities_and_nan(layout, variant):
    # IEEE specials in the operands: an infinite A entry makes its row +-inf
    # (NaN where it meets a zero of B), a NaN in B makes its column NaN.
    # Small-integer operands keep every finite output exact, so those are
    # compared bit for bit; NaN outputs are compared as a set (their sign
    # and payload are the hardware's).
    small = variant in KN_SKINNY + NK_SKINNY + [LDSB]
    M, N = (13, 264) if small else (300, 264)
    K = 1024 if variant == LDSB else 200
    A, B, Bt = int_operands(M, N, K, seed=31 + variant)
    A[3, 7] = float("inf")
    A[10, 20] = float("-inf")
    B[5, 9] = float("nan")
    Bt[9, 5] = float("nan")
    got = run_gemm(A, B, variant=variant) if layout == "kn" else run_gemm_bt(A, Bt, variant=variant)
    ref = oracle.gemm_bf16(A, B, M, N, K, b_layout="kn")
    nan_ref = _bf16_isnan(ref)
    assert nan_ref[:, 9].all() and nan_ref[3].any() and (ref[3] == 0x7F80).any() and (ref[10] == 0xFF80).any()
    assert np.array_equal(_bf16_isnan(got), nan_ref)
    assert np.array_equal(got[~nan_ref], ref[~nan_ref])


def test_gemm_tiled_variants_agree_bitwise():
    # every K x N tile accumulates each output over k in the same order
    A, B, _ = operands(384, 320, 448, seed=11)
    base = run_gemm(A, B, variant=KN_TILED[0])
    for v in KN_TILED[1:]:
        assert np.array_equal(run_gemm(A, B, variant=v), base), v


@pytest.mark.parametrize("variant", [0, 32, 35, 36, 37, 38, 39, 33])
def test_gemm_pad_and_grid_cap_do_not_change_result(variant):
    M = 16 if variant in KN_SKINNY else 520
    A, B, _ = operands(M, 384, 256, seed=5)
    base = run_gemm(A, B, variant=variant)
    for pad in (16 << 10, 64 << 10):
        plan = occ.occ_gemm_plan_query(M, 384, 256, pad, variant)
        if plan["feasible"]:
            assert np.array_equal(run_gemm(A, B, lds_bytes=pad, variant=variant), base), pad
    for cap in (1, 7, 256):
        assert np.array_equal(run_gemm(A, B, variant=variant, grid_cap=cap), base), cap


def test_gemm_identity_and_ones():
    A, _, _ = operands(96, 8, 128, seed=3)
    eye = torch.eye(128).to(torch.bfloat16)
    assert np.array_equal(run_gemm(A, eye), bf16_bits(A))
    ones_a = torch.ones((40, 512), dtype=torch.bfloat16)
    ones_b = torch.ones((512, 24), dtype=torch.bfloat16)
    assert np.all(run_gemm(ones_a, ones_b) == 0x4400)          # 512 in bf16


def test_gemm_empty_and_zero_k():
    assert run_gemm(torch.zeros((0, 64), dtype=torch.bfloat16),
                    torch.zeros((64, 16), dtype=torch.bfloat16)).shape == (0, 16)
    C = torch.full((20, 32), 1.0, device=DEV, dtype=torch.bfloat16)
    Ad = torch.zeros((20, 8), dtype=torch.bfloat16, device=DEV)[:, :0]
    assert occ.lib().occ_gemm(occ._ptr(Ad), None, occ._ptr(C), 20, 32, 0, 0, occ._stream(None)) == 0
    torch.cuda.synchronize()
    assert np.all(bf16_bits(C) == 0)                           # the empty sum is +0


def test_gemm_rejects_infeasible_pad_and_layout_mismatch():
    plan = occ.occ_gemm_plan_query(256, 256, 64, 0, 32)
    too_big = plan["max_lds_per_wg"] - plan["tile_lds_bytes"] + 16
    A, B, Bt = operands(64, 16, 64, seed=1)
    Ad, Bd, Btd = A.to(DEV), B.to(DEV), Bt.to(DEV)
    C = torch.empty((64, 16), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(occ.OccError) as e:
        occ.occ_gemm_ex(Ad, Bd, C, lds_bytes=too_big, variant=32)
    assert e.value.status == occ.OCC_ELDS
    for v in NK_TILED + NK_SKINNY + [LDSB]:                    # N x K variants
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_ex(Ad, Bd, C, variant=v)
        assert e.value.status == occ.OCC_EINVAL, v
    for v in KN_TILED + KN_SKINNY:                             # and the reverse
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_bt_ex(Ad, Btd, C, variant=v)
        assert e.value.status == occ.OCC_EINVAL, v
    A, B, _ = operands(64, 12, 64, seed=1)
    C = torch.empty((64, 12), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(occ.OccError) as e:                     # N % 8 != 0
        occ.occ_gemm(A.to(DEV), B.to(DEV), C)
    assert e.value.status == occ.OCC_EINVAL


def test_gemm_info_matches_plan():
    tile, max_wg, per_cu = occ.occ_gemm_info()
    p = occ.occ_gemm_plan_query(8192, 8192, 8192, 0, 32)
    assert (tile, max_wg, per_cu) == (p["tile_lds_bytes"], p["max_lds_per_wg"], p["lds_per_cu"])
    assert tile == 2 * 64 * (256 + 256) * 2 and per_cu == 160 * 1024 and max_wg >= tile
    assert occ.occ_gemm_plan_query(8192, 8192, 8192)["kernel_id"] == 32


def test_auto_choice_by_shape():
    # large: 256x256; mid: 128x128 three stages; small: the opt2 tile with
    # two stages; M <= 16: the skinny kernel
    assert occ.occ_gemm_plan_query(8192, 8192, 8192)["kernel_id"] == 32
    assert occ.occ_gemm_plan_query(2048, 2048, 4096)["kernel_id"] == 35
    assert occ.occ_gemm_plan_query(512, 512, 512)["kernel_id"] == 39
    assert occ.occ_gemm_plan_query(16, 28672, 8192)["kernel_id"] == 33
    assert occ.occ_gemm_plan_query(17, 28672, 8192)["kernel_id"] == 35    # 224 128x128 tiles
    assert occ.occ_gemm_bt_plan_query(8192, 8192, 8192)["kernel_id"] == 16
    assert occ.occ_gemm_bt_plan_query(2048, 2048, 4096)["kernel_id"] == 14
    assert occ.occ_gemm_bt_plan_query(512, 512, 512)["kernel_id"] == 9


def test_paper_tiles_lds_footprint():
    # Section 3.1: S_tile = 2 * (TILE_M * TILE_K + TILE_K * TILE_N) bytes for
    # the one-stage opt1 / opt2 tiles of Table 1
    for v, (tm, tn, tk) in ((OPT1_KN, (64, 64, 32)), (OPT2_KN, (64, 64, 64)), (6, (64, 64, 32)), (7, (64, 64, 64))):
        p = (occ.occ_gemm_plan_query if v in occ.KN_VARIANTS else occ.occ_gemm_bt_plan_query)(
            8192, 8192, 8192, 0, v)
        assert (p["tile_m"], p["tile_n"], p["tile_k"]) == (tm, tn, tk)
        assert p["tile_lds_bytes"] == 2 * (tm * tk + tk * tn)


@pytest.mark.parametrize("variant", [OPT1_KN, OPT2_KN, 38, 35, 32, 7])
def test_occupancy_follows_the_lds_formula(variant):
    """Residency is non-increasing in the pad and, wherever LDS binds, equals
    floor(LDS per CU / (S_tile + pad)) (Section 3.1); elsewhere it is the
    pad-free residency."""
    query = occ.occ_gemm_plan_query if variant in occ.KN_VARIANTS else occ.occ_gemm_bt_plan_query
    free = query(8192, 8192, 8192, 0, variant)["wg_per_cu"]    # registers / wave slots
    assert free >= 1
    prev = None
    bound_seen = False
    for pad_kib in (0, 8, 16, 24, 32, 48, 64, 96, 128):
        p = query(8192, 8192, 8192, pad_kib << 10, variant)
        w = p["wg_per_cu"] if p["feasible"] else 0
        if prev is not None:
            assert w <= prev, pad_kib
        prev = w
        if p["feasible"]:
            lds = p["lds_per_cu"] // (p["tile_lds_bytes"] + (pad_kib << 10))
            assert w == min(free, lds), (variant, pad_kib, w, free, lds)
            bound_seen |= lds < free
        else:
            assert p["tile_lds_bytes"] + (pad_kib << 10) > p["max_lds_per_wg"]
    if variant in (OPT1_KN, OPT2_KN, 7):
        assert bound_seen            # the paper's small tiles do reach the LDS-bound regime


# ----------------------------------------------------- occ_gemm_bt (N x K)
@pytest.mark.parametrize("M,N,K", [(512, 512, 512), (300, 200, 136), (1, 1, 8), (17, 33, 64),
                                   (257, 129, 520), (64, 64, 32), (16, 1000, 1032), (5, 77, 256),
                                   (16, 1000, 2048), (7, 333, 6144), (3, 100, 5120)])
def test_gemm_bt_auto_full_parity(M, N, K):
    A, _, Bt = operands(M, N, K, seed=0)
    got = run_gemm_bt(A, Bt)
    ref = oracle.gemm_bf16(A, Bt, M, N, K, b_layout="nk")
    frac = assert_gemm_close(got, ref, 1.0, 1.0, K, "bt auto %dx%dx%d" % (M, N, K))
    assert frac < 0.05


@pytest.mark.parametrize("variant", NK_TILED + NK_SKINNY)
def test_gemm_bt_every_variant_ragged_and_integer_exact(variant):
    M = 16 if variant in NK_SKINNY else 300
    A, _, Bt = operands(M, 260, 200, seed=variant)
    got = run_gemm_bt(A, Bt, variant=variant)
    assert_gemm_close(got, oracle.gemm_bf16(A, Bt, M, 260, 200), 1.0, 1.0, 200, "bt variant %d" % variant)
    M = 13 if variant in NK_SKINNY else 197
    A, _, Bt = int_operands(M, 150, 512, seed=variant)
    assert np.array_equal(run_gemm_bt(A, Bt, variant=variant), oracle.gemm_bf16(A, Bt, M, 150, 512))


def test_gemm_bt_tiled_variants_agree_bitwise_and_match_kn():
    # same tiles, same k order in both layouts: bit-identical for M > 16
    A, B, Bt = operands(384, 320, 448, seed=11)
    base = run_gemm_bt(A, Bt, variant=NK_TILED[0])
    for v in NK_TILED[1:]:
        assert np.array_equal(run_gemm_bt(A, Bt, variant=v), base), v
    assert np.array_equal(run_gemm(A, B), base)


@pytest.mark.parametrize("variant", [0, 7, 9, 16, 21])
def test_gemm_bt_pad_and_grid_cap_do_not_change_result(variant):
    M = 16 if variant in NK_SKINNY else 520
    A, _, Bt = operands(M, 384, 256, seed=5)
    base = run_gemm_bt(A, Bt, variant=variant)
    for pad in (16 << 10, 64 << 10):
        if occ.occ_gemm_bt_plan_query(M, 384, 256, pad, variant)["feasible"]:
            assert np.array_equal(run_gemm_bt(A, Bt, lds_bytes=pad, variant=variant), base), pad
    for cap in (1, 7, 256):
        assert np.array_equal(run_gemm_bt(A, Bt, variant=variant, grid_cap=cap), base), cap


@pytest.mark.parametrize("M,N", [(16, 260), (1, 17), (13, 1000)])
def test_gemm_bt_skinny_ldsb_full_parity(M, N):
    for K in (1024, 3072, 8192):
        A, _, Bt = operands(M, N, K, seed=M + K)
        got = run_gemm_bt(A, Bt, variant=LDSB)
        ref = oracle.gemm_bf16(A, Bt, M, N, K)
        assert_gemm_close(got, ref, 1.0, 1.0, K, "variant %d %dx%dx%d" % (LDSB, M, N, K))


def test_gemm_bt_skinny_ldsb_integer_bit_exact_and_invariant():
    # grid caps make workgroups run several units, so the block stream crosses units
    A, _, Bt = int_operands(11, 1000, 2048, seed=34)
    base = run_gemm_bt(A, Bt, variant=LDSB)
    assert np.array_equal(base, oracle.gemm_bf16(A, Bt, 11, 1000, 2048))
    for cap in (1, 3, 7):
        assert np.array_equal(run_gemm_bt(A, Bt, variant=LDSB, grid_cap=cap), base), cap
    assert np.array_equal(run_gemm_bt(A, Bt, variant=LDSB, lds_bytes=32 << 10), base)


def test_gemm_bt_skinny_k_rules_and_choice():
    for K in (1032, 512, 1536, 9216):
        A, Bt = inputs.gemm_operands(16, 64, K, seed=1, device=DEV)
        C = torch.empty((16, 64), device=DEV, dtype=torch.bfloat16)
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_bt_ex(A, Bt, C, variant=LDSB)
        assert e.value.status == occ.OCC_EINVAL, K
    for K, v in ((1024, LDSB), (3072, LDSB), (8192, LDSB), (512, 21), (8200, 21), (9216, 21)):
        assert occ.occ_gemm_bt_plan_query(16, 64, K)["kernel_id"] == v, K
    A, Bt = inputs.gemm_operands(17, 64, 64, seed=2, device=DEV)
    C = torch.empty((17, 64), device=DEV, dtype=torch.bfloat16)
    for v in (21, LDSB):                                       # M > 16
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_bt_ex(A, Bt, C, variant=v)
        assert e.value.status == occ.OCC_EINVAL


def test_gemm_bt_direct_to_lds_k_limit():
    # 32-bit pass offsets: K above the tile's limit is refused by that
    # variant, and the automatic choice for such K is the 64x64 tile (for B
    # N x K beyond that tile's own limit, the register-staged opt2 tile)
    big = (1 << 25) + 8
    with pytest.raises(occ.OccError) as e:
        occ.occ_gemm_bt_plan_query(4096, 4096, big, 0, 16)
    assert e.value.status == occ.OCC_EINVAL
    assert occ.occ_gemm_bt_plan_query(4096, 4096, big)["kernel_id"] == 7
    assert occ.occ_gemm_bt_plan_query(4096, 4096, 1 << 20)["kernel_id"] == 16
    assert occ.occ_gemm_plan_query(4096, 4096, (1 << 22) + 8)["kernel_id"] == 39
    assert occ.occ_gemm_bt_plan_query(4096, 4096, (1 << 22) + 8)["kernel_id"] == 9


def test_gemm_at_the_direct_to_lds_k_limit():
    """K at the 256x256 tile's limit, 2^22: one operand tile spans 2^31 bytes
    of 32-bit offsets.  Variant 32 (B K x N), variant 16 (B N x K) and the
    automatic choice agree bit for bit, and sampled 4 x 4 blocks (corners
    and the middle) match the oracle; K + 8 is refused by the 256-wide tiles."""
    M = N = 256
    K = 1 << 22
    assert occ.occ_gemm_plan_query(M, N, K, 0, 32)["kernel_id"] == 32
    with pytest.raises(occ.OccError) as e:
        occ.occ_gemm_plan_query(M, N, K + 8, 0, 32)
    assert e.value.status == occ.OCC_EINVAL
    A, Bt = inputs.gemm_operands(M, N, K, seed=9, device=DEV)
    B = Bt.t().contiguous()
    C32 = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    C16 = torch.empty_like(C32)
    Cauto = torch.empty_like(C32)
    occ.occ_gemm_ex(A, B, C32, variant=32)
    occ.occ_gemm_bt_ex(A, Bt, C16, variant=16)
    occ.occ_gemm(A, B, Cauto)
    torch.cuda.synchronize()
    assert torch.equal(C32.view(torch.int16), C16.view(torch.int16))
    assert torch.equal(C32.view(torch.int16), Cauto.view(torch.int16))
    del Bt, C16, Cauto
    Ah, Bh, Ch = bf16_bits(A), bf16_bits(B), bf16_bits(C32)
    for r0 in (0, 126, 252):
        for c0 in (0, 130, 252):
            ref = oracle.gemm_bf16(Ah, Bh, M, N, K, b_layout="kn", rows=(r0, r0 + 4), cols=(c0, c0 + 4))
            assert_gemm_close(Ch[r0:r0 + 4, c0:c0 + 4], ref, 1.0, 1.0, K, "K=2^22 block %d,%d" % (r0, c0))


def test_gemm_kn_at_its_n_limit():
    """B stored K x N at the 256x256 tile's N limit, 2^24 columns: a k-step's
    rows of B span 2^31 bytes of 32-bit offsets.  Variant 32 agrees bit for
    bit with the N x K kernel on the transposed B in sampled column blocks
    (the last columns included), and both match the oracle there; N + 8 is
    refused by variant 32."""
    M, N, K = 256, 1 << 24, 64
    assert occ.occ_gemm_plan_query(M, N, K, 0, 32)["kernel_id"] == 32
    with pytest.raises(occ.OccError) as e:
        occ.occ_gemm_plan_query(M, N + 8, K, 0, 32)
    assert e.value.status == occ.OCC_EINVAL
    A, Bt = inputs.gemm_operands(M, N, K, seed=11, device=DEV)
    B = Bt.t().contiguous()
    C32 = torch.empty((M, N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm_ex(A, B, C32, variant=32)
    C16 = torch.empty_like(C32)
    occ.occ_gemm_bt_ex(A, Bt, C16, variant=16)
    torch.cuda.synchronize()
    del Bt
    Ah, Bh = bf16_bits(A), bf16_bits(B)
    for c0 in (0, 4104, N // 2 + 12, N - 4):
        blk32 = C32[:, c0:c0 + 4].contiguous()
        assert torch.equal(blk32.view(torch.int16), C16[:, c0:c0 + 4].contiguous().view(torch.int16)), c0
        got = bf16_bits(blk32)
        for r0 in (0, 252):
            ref = oracle.gemm_bf16(Ah, Bh, M, N, K, b_layout="kn", rows=(r0, r0 + 4), cols=(c0, c0 + 4))
            assert_gemm_close(got[r0:r0 + 4], ref, 1.0, 1.0, K, "N=2^24 block %d,%d" % (r0, c0))


# ------------------------------------------------------------ skinny K x N
@pytest.mark.parametrize("M", [1, 5, 16])
@pytest.mark.parametrize("N,K", [(8, 8), (136, 40), (1000, 1032), (4104, 4096), (264, 8200), (128, 32)])
def test_gemm_skinny_full_parity(M, N, K):
    # ragged N (partial 128-column unit), K not a multiple of the 32-row
    # block or of the 4-wave split, fewer blocks than waves
    A, B, _ = operands(M, N, K, seed=M + N + K)
    got = run_gemm(A, B, variant=33)
    ref = oracle.gemm_bf16(A, B, M, N, K, b_layout="kn")
    assert_gemm_close(got, ref, 1.0, 1.0, K, "skinny %dx%dx%d" % (M, N, K))


def test_gemm_skinny_integer_bit_exact_invariant_and_bounded_reads():
    A, B, _ = int_operands(13, 1160, 2056, seed=12)
    base = run_gemm(A, B, variant=33)
    assert np.array_equal(base, oracle.gemm_bf16(A, B, 13, 1160, 2056, b_layout="kn"))
    for cap in (1, 3, 7):
        assert np.array_equal(run_gemm(A, B, variant=33, grid_cap=cap), base), cap
    assert np.array_equal(run_gemm(A, B, variant=33, lds_bytes=64 << 10), base)
    # a value a k-block past K would change the sum: nothing past K is read
    A2, B2, _ = int_operands(16, 256, 48, seed=13)
    big = torch.cat([B2, torch.full((16, 256), 2.0, dtype=torch.bfloat16)])
    C = torch.full((16, 256), float("nan"), device=DEV, dtype=torch.bfloat16)
    Ad, Bd = A2.to(DEV), big.to(DEV)                    # B has 64 rows; K = 48 uses 48
    assert occ.lib().occ_gemm_ex(occ._ptr(Ad), occ._ptr(Bd), occ._ptr(C), 16, 256, 48, 0, 33, 0,
                                 occ._stream(None)) == occ.OCC_OK
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(C), oracle.gemm_bf16(A2, B2, 16, 256, 48, b_layout="kn"))


def test_gemm_skinny_plan():
    p = occ.occ_gemm_plan_query(16, 28672, 8192)
    assert p["kernel_id"] == 33 and p["tile_n"] == 128 and p["tiles"] == 224
    assert p["grid"] == min(224, 2 * p["num_cus"]) and p["wg_per_cu"] >= 1
    A, B, _ = operands(17, 64, 64, seed=2)
    C = torch.empty((17, 64), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(occ.OccError) as e:              # M > 16
        occ.occ_gemm_ex(A.to(DEV), B.to(DEV), C, variant=33)
    assert e.value.status == occ.OCC_EINVAL


# ----------------------------------------------------------------- full sizes
def _check_sampled(A, B, C, M, N, K, layout, what, count=32, std_b=1.0):
    Ah, Bh, Ch = bf16_bits(A), bf16_bits(B), bf16_bits(C)
    for m0, n0 in sample_tiles(M, N, count=count):
        m1, n1 = min(m0 + 64, M), min(n0 + 64, N)
        ref = oracle.gemm_bf16(Ah, Bh, M, N, K, b_layout=layout, rows=(m0, m1), cols=(n0, n1))
        assert_gemm_close(Ch[m0:m1, n0:n1], ref, 1.0, std_b, K, "%s tile %d,%d" % (what, m0, n0))


@pytest.mark.parametrize("name", ["cb", "a2a", "paper_mb_ar"])
def test_gemm_full_size_sampled_tiles(name):
    """32 seeded 64x64 tiles, the four corners included, of the workload's
    full-size GEMM through occ_gemm; paper_mb_ar is Table 1's mb shape
    (8192 x 57344 x 8192)."""
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS[name]
    A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, device=DEV)
    B = Bt.t().contiguous()
    del Bt
    C = torch.empty((w.M, w.N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm(A, B, C)
    torch.cuda.synchronize()
    _check_sampled(A, B, C, w.M, w.N, w.K, "kn", name)


def test_gemm_full_size_layouts_agree_cb():
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS["cb"]
    A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, device=DEV)
    C_nk = torch.empty((w.M, w.N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm_bt(A, Bt, C_nk)
    B = Bt.t().contiguous()
    C = torch.empty_like(C_nk)
    occ.occ_gemm(A, B, C)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_nk.view(torch.int16))
    _check_sampled(A, Bt, C_nk, w.M, w.N, w.K, "nk", "cb bt", count=12)


def test_gemm_full_size_skinny_full_parity():
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS["mb"]
    A, Bt = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_b=w.std_b, seed_b=w.seed_b, device=DEV)
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(Bt), w.M, w.N, w.K)
    for v in (0, 21, LDSB):
        C = torch.full((w.M, w.N), float("nan"), device=DEV, dtype=torch.bfloat16)
        occ.occ_gemm_bt_ex(A, Bt, C, variant=v)
        torch.cuda.synchronize()
        assert_gemm_close(bf16_bits(C), ref, 1.0, w.std_b, w.K, "mb full, bt variant %d" % v)
    B = Bt.t().contiguous()
    for v in (0, 33, 32):
        C = torch.full((w.M, w.N), float("nan"), device=DEV, dtype=torch.bfloat16)
        occ.occ_gemm_ex(A, B, C, variant=v)
        torch.cuda.synchronize()
        assert_gemm_close(bf16_bits(C), ref, 1.0, w.std_b, w.K, "mb full, variant %d" % v)
