"""GEMM parity: the HIP kernels (through the C ABI) against the CPU oracle."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_09200_amd import binding as occ
from paper_2606_09200_amd import inputs
from gpu_common import DEV, assert_gemm_close, bf16_bits, sample_tiles

pytestmark = pytest.mark.gpu

TILED = [1, 2, 3, 4, 5, 6, 7, 9, 10, 11, 12, 13, 14, 15, 16, 17, 18, 19, 24, 25, 26, 27]
SKINNY = [8, 20, 21, 22, 23]
AREG = {28: 8192, 29: 4096}   # skinny with A in registers: largest K (K % 2048 == 0)
LDSB = 34                     # skinny, A in registers, B through LDS: K % 1024 == 0, K <= 8192


def run_gemm(A, B, lds_bytes=0, variant=0, grid_cap=0):
    M, K = A.shape
    N = B.shape[0]
    Ad, Bd = A.to(DEV), B.to(DEV)
    C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm_ex(Ad, Bd, C, lds_bytes=lds_bytes, variant=variant, grid_cap=grid_cap)
    torch.cuda.synchronize()
    return bf16_bits(C)


def int_operands(M, N, K, seed):
    g = torch.Generator().manual_seed(seed)
    A = torch.randint(-2, 3, (M, K), generator=g).to(torch.bfloat16)
    B = torch.randint(-2, 3, (N, K), generator=g).to(torch.bfloat16)
    return A, B


@pytest.mark.parametrize("M,N,K", [(512, 512, 512), (300, 200, 136), (1, 1, 8), (17, 33, 64),
                                   (257, 129, 520), (64, 64, 32), (16, 1000, 1032), (5, 77, 256),
                                   (16, 1000, 2048), (7, 333, 6144), (3, 100, 5120)])
def test_gemm_auto_full_parity(M, N, K):
    A, B = inputs.gemm_operands(M, N, K, seed=0)
    got = run_gemm(A, B)
    ref = oracle.gemm_bf16(A, B, M, N, K)
    frac = assert_gemm_close(got, ref, 1.0, 1.0, K, "auto %dx%dx%d" % (M, N, K))
    assert frac < 0.05


@pytest.mark.parametrize("variant", TILED + SKINNY)
def test_gemm_every_variant_ragged(variant):
    M = 16 if variant in SKINNY else 300
    N, K = 260, 200
    A, B = inputs.gemm_operands(M, N, K, seed=variant)
    got = run_gemm(A, B, variant=variant)
    ref = oracle.gemm_bf16(A, B, M, N, K)
    assert_gemm_close(got, ref, 1.0, 1.0, K, "variant %d" % variant)


@pytest.mark.parametrize("variant", TILED + SKINNY)
def test_gemm_integer_operands_bit_exact(variant):
    # sums of products of {-2..2} are exact in fp32 in any order: bit-exact
    M = 13 if variant in SKINNY else 197
    A, B = int_operands(M, 150, 512, seed=variant)
    got = run_gemm(A, B, variant=variant)
    assert np.array_equal(got, oracle.gemm_bf16(A, B, M, 150, 512))


@pytest.mark.parametrize("variant", sorted(AREG))
@pytest.mark.parametrize("M,N", [(16, 260), (1, 17), (13, 1000)])
def test_gemm_skinny_areg_full_parity(variant, M, N):
    for K in range(2048, AREG[variant] + 1, 2048):
        A, B = inputs.gemm_operands(M, N, K, seed=variant + K)
        got = run_gemm(A, B, variant=variant)
        ref = oracle.gemm_bf16(A, B, M, N, K)
        assert_gemm_close(got, ref, 1.0, 1.0, K, "variant %d %dx%dx%d" % (variant, M, N, K))


@pytest.mark.parametrize("variant", sorted(AREG))
def test_gemm_skinny_areg_integer_bit_exact_and_invariant(variant):
    A, B = int_operands(11, 150, 2048, seed=variant)
    base = run_gemm(A, B, variant=variant)
    assert np.array_equal(base, oracle.gemm_bf16(A, B, 11, 150, 2048))
    for cap in (1, 7):
        assert np.array_equal(run_gemm(A, B, variant=variant, grid_cap=cap), base), cap
    assert np.array_equal(run_gemm(A, B, variant=variant, lds_bytes=32 << 10), base)


@pytest.mark.parametrize("variant", sorted(AREG))
def test_gemm_skinny_areg_rejects_unsupported_k(variant):
    for K in (1032, 512, 1024, 3072, AREG[variant] + 2048):
        A, B = inputs.gemm_operands(16, 64, K, seed=1, device=DEV)
        C = torch.empty((16, 64), device=DEV, dtype=torch.bfloat16)
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_ex(A, B, C, variant=variant)
        assert e.value.status == occ.OCC_EINVAL, K
    with pytest.raises(occ.OccError):
        occ.occ_gemm_plan_query(16, 64, 0, 0, variant)          # K = 0: not this kernel
    for K, v in ((1024, LDSB), (3072, LDSB), (4096, LDSB), (8192, LDSB), (512, 21), (8200, 21), (9216, 21)):
        assert occ.occ_gemm_plan_query(16, 64, K, 0, 0)["kernel_id"] == v, K


@pytest.mark.parametrize("M,N", [(16, 260), (1, 17), (13, 1000)])
def test_gemm_skinny_ldsb_full_parity(M, N):
    for K in (1024, 3072, 8192):
        A, B = inputs.gemm_operands(M, N, K, seed=M + K)
        got = run_gemm(A, B, variant=LDSB)
        ref = oracle.gemm_bf16(A, B, M, N, K)
        assert_gemm_close(got, ref, 1.0, 1.0, K, "variant %d %dx%dx%d" % (LDSB, M, N, K))


def test_gemm_skinny_ldsb_integer_bit_exact_and_invariant():
    # sums of products of {-2..2} are exact in fp32 in any order; grid caps
    # make workgroups run several units, so the block stream crosses units
    A, B = int_operands(11, 1000, 2048, seed=34)
    base = run_gemm(A, B, variant=LDSB)
    assert np.array_equal(base, oracle.gemm_bf16(A, B, 11, 1000, 2048))
    for cap in (1, 3, 7):
        assert np.array_equal(run_gemm(A, B, variant=LDSB, grid_cap=cap), base), cap
    assert np.array_equal(run_gemm(A, B, variant=LDSB, lds_bytes=32 << 10), base)


def test_gemm_skinny_ldsb_rejects_unsupported_k():
    for K in (1032, 512, 1536, 9216):
        A, B = inputs.gemm_operands(16, 64, K, seed=1, device=DEV)
        C = torch.empty((16, 64), device=DEV, dtype=torch.bfloat16)
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_ex(A, B, C, variant=LDSB)
        assert e.value.status == occ.OCC_EINVAL, K
    with pytest.raises(occ.OccError):
        occ.occ_gemm_plan_query(16, 64, 0, 0, LDSB)


def test_gemm_direct_to_lds_k_limit():
    # 32-bit pass offsets: K above the variant's limit is refused, and the
    # automatic choice for such K is a register-staged variant (plan only)
    big = (1 << 25) + 8
    with pytest.raises(occ.OccError) as e:
        occ.occ_gemm_plan_query(4096, 4096, big, 0, 16)
    assert e.value.status == occ.OCC_EINVAL
    assert occ.occ_gemm_plan_query(4096, 4096, big)["kernel_id"] == 3
    assert occ.occ_gemm_plan_query(4096, 4096, 1 << 20)["kernel_id"] == 16


def test_gemm_identity_and_ones():
    A, _ = inputs.gemm_operands(96, 8, 128, seed=3)
    eye = torch.eye(128).to(torch.bfloat16)
    assert np.array_equal(run_gemm(A, eye), bf16_bits(A))
    ones_a = torch.ones((40, 512), dtype=torch.bfloat16)
    ones_b = torch.ones((24, 512), dtype=torch.bfloat16)
    assert np.all(run_gemm(ones_a, ones_b) == 0x4400)


def test_gemm_tiled_variants_agree_bitwise():
    A, B = inputs.gemm_operands(384, 320, 448, seed=11)
    base = run_gemm(A, B, variant=1)
    for v in TILED[1:]:
        assert np.array_equal(run_gemm(A, B, variant=v), base), v


@pytest.mark.parametrize("variant", [0, 1, 5, 7, 8, 10, 16, 17, 20, 23])
def test_gemm_pad_and_grid_cap_do_not_change_result(variant):
    M = 16 if variant in SKINNY else 520
    A, B = inputs.gemm_operands(M, 384, 256, seed=5)
    base = run_gemm(A, B, variant=variant)
    for pad in (16 << 10, 64 << 10):
        plan = occ.occ_gemm_plan_query(M, 384, 256, pad, variant)
        if plan["feasible"]:
            assert np.array_equal(run_gemm(A, B, lds_bytes=pad, variant=variant), base), pad
    for cap in (1, 7, 256):
        assert np.array_equal(run_gemm(A, B, variant=variant, grid_cap=cap), base), cap


def test_gemm_empty_and_zero_k():
    A = torch.zeros((0, 64), dtype=torch.bfloat16)
    B = torch.zeros((32, 64), dtype=torch.bfloat16)
    assert run_gemm(A, B).shape == (0, 32)
    A = torch.zeros((20, 0), dtype=torch.bfloat16)
    B = torch.zeros((30, 0), dtype=torch.bfloat16)
    Ad = torch.zeros((20, 8), dtype=torch.bfloat16, device=DEV)[:, :0]
    C = torch.full((20, 30), 1.0, device=DEV, dtype=torch.bfloat16)
    occ.lib().occ_gemm(occ._ptr(Ad), None, occ._ptr(C), 20, 30, 0, 0, occ._stream(None))
    torch.cuda.synchronize()
    assert np.all(bf16_bits(C) == 0)


def test_gemm_rejects_infeasible_pad():
    A, B = inputs.gemm_operands(256, 256, 64, seed=1)
    plan = occ.occ_gemm_plan_query(256, 256, 64, 0, 1)
    too_big = plan["max_lds_per_wg"] - plan["tile_lds_bytes"] + 16
    C = torch.empty((256, 256), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(occ.OccError) as e:
        occ.occ_gemm_ex(A.to(DEV), B.to(DEV), C, lds_bytes=too_big, variant=1)
    assert e.value.status == occ.OCC_ELDS


def test_gemm_info_matches_plan():
    tile, max_wg, per_cu = occ.occ_gemm_info()
    p = occ.occ_gemm_plan_query(8192, 8192, 8192, 0, 16)
    assert (tile, max_wg, per_cu) == (p["tile_lds_bytes"], p["max_lds_per_wg"], p["lds_per_cu"])
    assert tile == 2 * 64 * (256 + 256) * 2 and per_cu == 160 * 1024 and max_wg >= tile


def test_occupancy_non_increasing_in_pad():
    for variant in (0, 5, 6, 7):
        prev = None
        for pad_kib in (0, 16, 32, 64, 96, 128):
            p = occ.occ_gemm_plan_query(8192, 8192, 8192, pad_kib << 10, variant)
            w = p["wg_per_cu"] if p["feasible"] else 0
            if prev is not None:
                assert w <= prev
            prev = w
            if p["feasible"]:
                # where LDS binds, residency is floor(LDS per CU / (S_tile + pad))
                lds_bound = p["lds_per_cu"] // (p["tile_lds_bytes"] + (pad_kib << 10))
                assert w <= lds_bound


# ----------------------------------------------------------------- full sizes
@pytest.mark.parametrize("name", ["cb", "a2a"])
def test_gemm_full_size_sampled_tiles(name):
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS[name]
    A, B = inputs.gemm_operands(w.M, w.N, w.K, seed=0, device=DEV)
    C = torch.empty((w.M, w.N), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm(A, B, C)
    torch.cuda.synchronize()
    Ah, Bh, Ch = bf16_bits(A), bf16_bits(B), bf16_bits(C)
    for m0, n0 in sample_tiles(w.M, w.N):
        m1, n1 = min(m0 + 64, w.M), min(n0 + 64, w.N)
        ref = oracle.gemm_bf16(Ah, Bh, w.M, w.N, w.K, rows=(m0, m1), cols=(n0, n1))
        assert_gemm_close(Ch[m0:m1, n0:n1], ref, 1.0, 1.0, w.K, "%s tile %d,%d" % (name, m0, n0))


def test_gemm_full_size_skinny_full_parity():
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS["mb"]
    A, B = inputs.gemm_operands(w.M, w.N, w.K, seed=0, std_b=w.std_b, seed_b=w.seed_b, device=DEV)
    ref = oracle.gemm_bf16(bf16_bits(A), bf16_bits(B), w.M, w.N, w.K)
    for v in [0] + SKINNY + [28, LDSB]:
        C = torch.full((w.M, w.N), float("nan"), device=DEV, dtype=torch.bfloat16)
        occ.occ_gemm_ex(A, B, C, variant=v)
        torch.cuda.synchronize()
        assert_gemm_close(bf16_bits(C), ref, 1.0, w.std_b, w.K, "mb full, variant %d" % v)
    # B stored K x N: the skinny K x N kernel (automatic) and the 256x256 tile
    Bkn = B.t().contiguous()
    for v in (0, 33, 32):
        C = torch.full((w.M, w.N), float("nan"), device=DEV, dtype=torch.bfloat16)
        occ.occ_gemm_kn_ex(A, Bkn, C, variant=v)
        torch.cuda.synchronize()
        assert_gemm_close(bf16_bits(C), ref, 1.0, w.std_b, w.K, "mb full, K x N, variant %d" % v)


# ------------------------------------------------------------- B stored K x N
def run_gemm_kn(A, Bkn, lds_bytes=0, variant=0, grid_cap=0):
    M, K = A.shape
    N = Bkn.shape[1]
    Ad, Bd = A.to(DEV), Bkn.to(DEV)
    C = torch.full((M, N), float("nan"), device=DEV, dtype=torch.bfloat16)
    occ.occ_gemm_kn_ex(Ad, Bd, C, lds_bytes=lds_bytes, variant=variant, grid_cap=grid_cap)
    torch.cuda.synchronize()
    return bf16_bits(C)


@pytest.mark.parametrize("M,N,K", [(512, 512, 512), (300, 264, 136), (1, 8, 8), (17, 40, 64),
                                   (257, 136, 520), (64, 64, 32), (520, 1000, 1032),
                                   (16, 256, 4096), (600, 776, 200)])
def test_gemm_kn_full_parity(M, N, K):
    A, B = inputs.gemm_operands(M, N, K, seed=4)
    Bkn = B.t().contiguous()
    got = run_gemm_kn(A, Bkn)
    ref = oracle.gemm_bf16(A, Bkn, M, N, K, b_layout="kn")
    assert_gemm_close(got, ref, 1.0, 1.0, K, "kn %dx%dx%d" % (M, N, K))
    if M > 16:
        # the same tile, MFMA sequence and k order as the N x K kernel: same bits
        assert np.array_equal(got, run_gemm(A, B, variant=16))
    else:
        # the skinny K x N kernel (automatic for M <= 16)
        assert occ.occ_gemm_plan_query(M, N, K, b_layout="kn")["kernel_id"] == 33
        assert np.array_equal(got, run_gemm_kn(A, Bkn, variant=33))


def test_gemm_kn_integer_bit_exact_and_invariant():
    A, B = int_operands(333, 272, 712, seed=9)
    Bkn = B.t().contiguous()
    base = run_gemm_kn(A, Bkn)
    assert np.array_equal(base, oracle.gemm_bf16(A, Bkn, 333, 272, 712, b_layout="kn"))
    for cap in (1, 3, 256):
        assert np.array_equal(run_gemm_kn(A, Bkn, grid_cap=cap), base), cap
    assert np.array_equal(run_gemm_kn(A, Bkn, lds_bytes=16 << 10, variant=32), base)


@pytest.mark.parametrize("M", [1, 5, 16])
@pytest.mark.parametrize("N,K", [(8, 8), (136, 40), (1000, 1032), (4104, 4096), (264, 8200), (128, 32)])
def test_gemm_kn_skinny_full_parity(M, N, K):
    # ragged N (partial 128-column unit), K not a multiple of the 32-row
    # block or of the 4-wave split, fewer blocks than waves
    A, B = inputs.gemm_operands(M, N, K, seed=M + N + K)
    Bkn = B.t().contiguous()
    got = run_gemm_kn(A, Bkn, variant=33)
    ref = oracle.gemm_bf16(A, Bkn, M, N, K, b_layout="kn")
    assert_gemm_close(got, ref, 1.0, 1.0, K, "kn skinny %dx%dx%d" % (M, N, K))


def test_gemm_kn_skinny_integer_bit_exact_and_invariant():
    # sums of products of {-2..2} are exact in fp32 in any order
    A, B = int_operands(13, 1160, 2056, seed=12)
    Bkn = B.t().contiguous()
    base = run_gemm_kn(A, Bkn, variant=33)
    assert np.array_equal(base, oracle.gemm_bf16(A, Bkn, 13, 1160, 2056, b_layout="kn"))
    for cap in (1, 3, 7):
        assert np.array_equal(run_gemm_kn(A, Bkn, variant=33, grid_cap=cap), base), cap
    assert np.array_equal(run_gemm_kn(A, Bkn, variant=33, lds_bytes=64 << 10), base)
    # a value a k-block past K would change the sum: nothing past K is read
    A2, B2 = int_operands(16, 256, 48, seed=13)
    big = torch.cat([B2.t().contiguous(), torch.full((16, 256), 2.0, dtype=torch.bfloat16)])
    C = torch.full((16, 256), float("nan"), device=DEV, dtype=torch.bfloat16)
    Ad, Bd = A2.to(DEV), big.to(DEV)                    # B has 64 rows; K = 48 uses 48
    assert occ.lib().occ_gemm_kn_ex(occ._ptr(Ad), occ._ptr(Bd), occ._ptr(C), 16, 256, 48, 0, 33, 0,
                                    occ._stream(None)) == occ.OCC_OK
    torch.cuda.synchronize()
    assert np.array_equal(bf16_bits(C), oracle.gemm_bf16(A2, B2.t().contiguous(), 16, 256, 48, b_layout="kn"))


def test_gemm_kn_skinny_plan_and_checks():
    p = occ.occ_gemm_plan_query(16, 28672, 8192, b_layout="kn")
    assert p["kernel_id"] == 33 and p["tile_n"] == 128 and p["tiles"] == 224
    assert p["grid"] == min(224, 2 * p["num_cus"]) and p["wg_per_cu"] >= 1
    assert occ.occ_gemm_plan_query(17, 28672, 8192, b_layout="kn")["kernel_id"] == 32
    assert occ.occ_gemm_plan_query(16, 28672, 8192, 0, 33)["kernel_id"] == 33   # K x N from the id
    with pytest.raises(occ.OccError):                   # the K x N plan of an N x K variant
        occ.occ_gemm_plan_query(16, 64, 64, 0, 28, b_layout="kn")
    A, B = inputs.gemm_operands(17, 64, 64, seed=2, device=DEV)
    C = torch.empty((17, 64), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(occ.OccError) as e:              # M > 16
        occ.occ_gemm_kn_ex(A, B.t().contiguous(), C, variant=33)
    assert e.value.status == occ.OCC_EINVAL
    with pytest.raises(occ.OccError) as e:              # B read as N x K
        occ.occ_gemm_ex(A[:16], B, C[:16], variant=33)
    assert e.value.status == occ.OCC_EINVAL


def test_gemm_kn_layout_checks():
    A, B = inputs.gemm_operands(64, 12, 64, seed=1, device=DEV)
    Bkn = B.t().contiguous()
    C = torch.empty((64, 12), device=DEV, dtype=torch.bfloat16)
    with pytest.raises(occ.OccError) as e:            # N % 8 != 0
        occ.occ_gemm_kn(A, Bkn, C)
    assert e.value.status == occ.OCC_EINVAL
    A, B = inputs.gemm_operands(64, 16, 64, seed=1, device=DEV)
    Bkn = B.t().contiguous()
    C = torch.empty((64, 16), device=DEV, dtype=torch.bfloat16)
    for v in (1, 16, 21):                               # variants that read B as N x K
        with pytest.raises(occ.OccError) as e:
            occ.occ_gemm_kn_ex(A, Bkn, C, variant=v)
        assert e.value.status == occ.OCC_EINVAL, v
    with pytest.raises(occ.OccError) as e:              # and the reverse
        occ.occ_gemm_ex(A, B, C, variant=32)
    assert e.value.status == occ.OCC_EINVAL
    p = occ.occ_gemm_plan_query(8192, 8192, 8192, 0, 32)
    q = occ.occ_gemm_plan_query(8192, 8192, 8192, 0, 16)
    assert p["kernel_id"] == 32 and p["tile_lds_bytes"] == q["tile_lds_bytes"]
    assert (p["tile_m"], p["tile_n"], p["tile_k"], p["grid"]) == (q["tile_m"], q["tile_n"], q["tile_k"], q["grid"])
    assert p["wg_per_cu"] >= 1


def test_gemm_kn_zero_k_and_empty():
    C = torch.full((20, 32), 1.0, device=DEV, dtype=torch.bfloat16)
    Ad = torch.zeros((20, 8), dtype=torch.bfloat16, device=DEV)[:, :0]
    occ.lib().occ_gemm_kn(occ._ptr(Ad), None, occ._ptr(C), 20, 32, 0, 0, occ._stream(None))
    torch.cuda.synchronize()
    assert np.all(bf16_bits(C) == 0)
    A = torch.zeros((0, 64), dtype=torch.bfloat16)
    assert run_gemm_kn(A, torch.zeros((64, 16), dtype=torch.bfloat16)).shape == (0, 16)


def test_gemm_kn_full_size_sampled_and_equal_to_nk():
    from paper_2606_09200_amd.workloads import WORKLOADS
    w = WORKLOADS["cb"]
    A, B = inputs.gemm_operands(w.M, w.N, w.K, seed=0, device=DEV)
    Bkn = B.t().contiguous()
    C = torch.empty((w.M, w.N), device=DEV, dtype=torch.bfloat16)
    C_nk = torch.empty_like(C)
    occ.occ_gemm_kn(A, Bkn, C)
    occ.occ_gemm_ex(A, B, C_nk, variant=16)
    torch.cuda.synchronize()
    assert torch.equal(C.view(torch.int16), C_nk.view(torch.int16))
    Ah, Bh, Ch = bf16_bits(A), bf16_bits(Bkn), bf16_bits(C)
    for m0, n0 in sample_tiles(w.M, w.N, count=12):
        m1, n1 = min(m0 + 64, w.M), min(n0 + 64, w.N)
        ref = oracle.gemm_bf16(Ah, Bh, w.M, w.N, w.K, b_layout="kn", rows=(m0, m1), cols=(n0, n1))
        assert_gemm_close(Ch[m0:m1, n0:n1], ref, 1.0, 1.0, w.K, "cb kn tile %d,%d" % (m0, n0))
