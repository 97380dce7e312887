"""CPU checks of the C ABI: the library loads, exports every declared entry
point, and rejects bad arguments with the documented status before touching
the GPU.  The pointers here are placeholders, never device memory: a call
that passes validation would go on to launch kernels on them, so such calls
are made only where no device is visible (they then stop at the device
lookup with OCC_ENODEV), never on a machine with a GPU."""
import ctypes
import os
import re

import pytest

OCC_ENODEV = -6


def no_device(L):
    """True when the library's own device lookup finds no gfx950 device (the
    step every call takes right after validation)."""
    x = ctypes.c_int(0)
    return L.occ_gemm_info(ctypes.byref(x), ctypes.byref(x), ctypes.byref(x)) == OCC_ENODEV


def expect_accepted(L, call, *args):
    """``call(*args)`` passes validation: checked only without a device, where
    the next step (the device lookup) fails with OCC_ENODEV."""
    if no_device(L):
        assert call(*args) == OCC_ENODEV, args

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "occ.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    from paper_2606_09200_amd import binding
    return binding.lib()


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ("occ_gemm", "share_reduce", "share_permute", "run_overlap", "occ_strerror"):
        assert f in names


def test_library_exports_every_declared_symbol(L):
    missing = [f for f in declared_functions() if not hasattr(L, f)]
    assert not missing, missing


def test_strerror_and_version(L):
    from paper_2606_09200_amd import binding
    for code in range(0, -8, -1):
        assert binding.occ_strerror(code).startswith("OCC_")
    assert "unknown" in binding.occ_strerror(-99)
    assert binding.occ_version() == binding.ABI_VERSION == (2, 2)
    hdr = open(HEADER).read()
    assert "#define OCC_VERSION_MAJOR 2" in hdr and "#define OCC_VERSION_MINOR 2" in hdr


P = ctypes.c_void_p


def test_gemm_argument_errors(L):
    # occ_gemm takes B stored K x N: bad sizes, K or N not a multiple of 8,
    # null or misaligned pointers, aliasing
    assert L.occ_gemm(P(0x1000), P(0x2000), P(0x3000), -1, 8, 8, 0, None) == -1
    assert L.occ_gemm(P(0x1000), P(0x2000), P(0x3000), 4, 8, 12, 0, None) == -1
    assert L.occ_gemm(P(0x1000), P(0x2000), P(0x3000), 4, 12, 8, 0, None) == -1   # N % 8 (16-byte B rows)
    assert L.occ_gemm(None, P(0x2000), P(0x3000), 4, 8, 8, 0, None) == -1
    assert L.occ_gemm(P(0x1000), None, P(0x3000), 4, 8, 8, 0, None) == -1
    assert L.occ_gemm(P(0x1008), P(0x2000), P(0x3000), 4, 8, 8, 0, None) == -1
    assert L.occ_gemm(P(0x1000), P(0x2000), P(0x1010), 4, 8, 8, 0, None) == -4     # C inside A
    assert L.occ_gemm(P(0x1000), P(0x2000), P(0x2010), 4, 8, 8, 0, None) == -4     # C inside B
    assert L.occ_gemm_ex(P(0x1000), P(0x2000), P(0x3000), 4, 8, 8, 0, -1, 0, None) == -1
    assert L.occ_gemm_ex(P(0x1000), P(0x2000), P(0x3000), 4, 8, 8, 0, 0, -5, None) == -1


def test_gemm_bt_argument_errors(L):
    # occ_gemm_bt takes B stored N x K: the same checks except N % 8
    assert L.occ_gemm_bt(P(0x1000), P(0x2000), P(0x3000), 4, 4, 12, 0, None) == -1
    assert L.occ_gemm_bt(None, P(0x2000), P(0x3000), 4, 4, 8, 0, None) == -1
    assert L.occ_gemm_bt(P(0x1000), P(0x2000), P(0x1010), 4, 4, 8, 0, None) == -4  # C inside A
    assert L.occ_gemm_bt_ex(P(0x1000), P(0x2000), P(0x3000), 4, 4, 8, 0, -1, 0, None) == -1
    assert L.occ_gemm_bt_ex(P(0x1000), P(0x2000), P(0x3000), 4, 4, 8, 0, 0, -1, None) == -1
    # N % 8 != 0 is fine for the N x K layout (fails later, with no device)
    expect_accepted(L, L.occ_gemm_bt, P(0x1000), P(0x2000), P(0x3000), 4, 12, 8, 0, None)


def test_gemm_plan_query_argument_errors(L):
    from paper_2606_09200_amd import binding
    plan = binding.occ_gemm_plan()
    for q in (L.occ_gemm_plan_query, L.occ_gemm_bt_plan_query):
        assert q(16, 64, 64, 0, 0, 0, None) == -1
        assert q(-1, 64, 64, 0, 0, 0, ctypes.byref(plan)) == -1
        assert q(16, 64, 64, 0, -1, 0, ctypes.byref(plan)) == -1
        assert q(16, 64, 64, 0, 0, -1, ctypes.byref(plan)) == -1
    with pytest.raises(ValueError):
        binding.occ_gemm_plan_query(16, 64, 64, b_layout="nn")


def test_binding_variant_tables_match_header():
    """Every variant id the header names is in the binding's table of its
    layout, and nothing else is."""
    from paper_2606_09200_amd import binding
    text = open(HEADER).read()
    enum = text[text.index("OCC_GEMM_AUTO = 0"):]
    enum = enum[:enum.index("};")]
    kn = {int(v) for v in re.findall(r"OCC_GEMM_KN_\w+ = (\d+)", enum)}
    ids = {int(v) for v in re.findall(r"OCC_GEMM_\w+ = (\d+)", enum)} - {0}
    assert kn == set(binding.KN_VARIANTS)
    assert ids - kn == set(binding.NK_VARIANTS)
    assert set(binding.SKINNY_VARIANTS) <= ids


def test_reduce_argument_errors(L):
    arr = (ctypes.c_void_p * 65)(*([0x10000 * (i + 1) for i in range(65)]))
    out = P(0x900000)
    assert L.share_reduce(arr, 0, 16, out, None) == -1
    assert L.share_reduce(arr, 65, 16, out, None) == -1
    assert L.share_reduce(None, 2, 16, out, None) == -1
    assert L.share_reduce(arr, 2, 16, None, None) == -1
    assert L.share_reduce(arr, 2, 16, P(0x10000 + 8), None) == -4      # out overlaps chunk 0
    nul = (ctypes.c_void_p * 2)(0x10000, 0)
    assert L.share_reduce(nul, 2, 16, out, None) == -1
    odd = (ctypes.c_void_p * 2)(0x10002, 0x20000)
    assert L.share_reduce(odd, 2, 16, out, None) == -1                # not 4-byte aligned
    assert L.share_reduce_ex(arr, 2, 16, out, 0, 4, None) == -1       # priority out of range
    assert L.share_reduce_ex(arr, 2, 16, out, -1, 0, None) == -1


def test_reduce_own_argument_errors(L):
    arr = (ctypes.c_void_p * 64)(*([0x100000 * (i + 1) for i in range(64)]))
    own, out = P(0x9000000), P(0xA000000)
    assert L.share_reduce_own(own, arr, -1, 16, out, 0, 0, None) == -1
    assert L.share_reduce_own(own, arr, 64, 16, out, 0, 0, None) == -1        # 1 + 64 terms
    assert L.share_reduce_own(own, None, 2, 16, out, 0, 0, None) == -1
    assert L.share_reduce_own(None, arr, 2, 16, out, 0, 0, None) == -1
    assert L.share_reduce_own(P(0x9000001), arr, 2, 16, out, 0, 0, None) == -1  # own not 2-byte aligned
    assert L.share_reduce_own(own, arr, 2, 16, P(0x9000000 + 8), 0, 0, None) == -4  # out over own
    assert L.share_reduce_own(own, arr, 2, 16, P(0x100000 + 4), 0, 0, None) == -4   # out over a peer
    assert L.share_reduce_own(own, arr, 2, 16, out, 0, 4, None) == -1         # priority
    assert L.share_reduce_own(own, arr, 2, 16, out, -1, 0, None) == -1
    assert L.share_reduce_own(own, None, 0, 0, out, 0, 0, None) == 0          # len 0: no-op
    # valid arguments pass validation (and then need a device)
    expect_accepted(L, L.share_reduce_own, own, None, 0, 16, out, 0, 0, None)


def test_permute_argument_errors(L):
    perm = (ctypes.c_int32 * 4)(0, 2, 2, 3)
    assert L.share_permute(P(0x1000), P(0x100000), perm, 4, 64, None) == -3
    perm = (ctypes.c_int32 * 4)(0, 1, 4, 3)
    assert L.share_permute(P(0x1000), P(0x100000), perm, 4, 64, None) == -3
    perm = (ctypes.c_int32 * 4)(3, 1, 0, 2)
    assert L.share_permute(P(0x1000), P(0x1000 + 128), perm, 4, 64, None) == -4
    assert L.share_permute(None, P(0x100000), perm, 4, 64, None) == -1
    assert L.share_permute(P(0x1000), P(0x100000), None, 4, 64, None) == -1
    assert L.share_permute(P(0x1000), P(0x100000), perm, 0, 64, None) == -1
    assert L.share_permute(P(0x1000), P(0x100000), perm, 513, 64, None) == -1


def test_run_overlap_argument_errors(L):
    from paper_2606_09200_amd import binding as b
    cfg = b.occ_overlap_cfg()
    res = b.occ_overlap_result()
    assert L.run_overlap(None, ctypes.byref(res)) == -1
    assert L.run_overlap(ctypes.byref(cfg), None) == -1
    cfg.M = cfg.N = cfg.K = 8
    cfg.A, cfg.B, cfg.C = 0x1000, 0x2000, 0x3000
    arr = (ctypes.c_void_p * 2)(0x10000, 0x20000)
    cfg.bufs = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    cfg.nchunks, cfg.len, cfg.out = 2, 64, 0x30000
    cfg.n_iter, cfg.reps, cfg.warmup = 0, 1, 0
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1   # n_iter < 1
    cfg.n_iter = 2
    cfg.comm_priority = 7
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.comm_priority = 3
    cfg.comm_kind = 5
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.comm_kind = 0
    cfg.out = 0x3000 + 16                                                 # comm output inside C
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -4
    cfg.out = 0x30000
    arr2 = (ctypes.c_void_p * 2)(0x10000, 0x3000)                         # C is a comm input
    cfg.bufs = ctypes.cast(arr2, ctypes.POINTER(ctypes.c_void_p))
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -4
    cfg.bufs = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    cfg.flags = 64
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.flags = 16                                                        # OCC_RUN_PACE_ALL is valid
    expect_accepted(L, L.run_overlap, ctypes.byref(cfg), ctypes.byref(res))
    cfg.flags = 0
    cfg.gemm_b_layout = 2                                                 # neither K x N nor N x K
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.gemm_b_layout = 0
    cfg.dep = 2                                                           # neither event nor counter
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.dep, cfg.n_iter = 1, 1025                                         # counters for 1024 iterations
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.n_iter = 2
    expect_accepted(L, L.run_overlap, ctypes.byref(cfg), ctypes.byref(res))
    cfg.flags = 8 | 2                                                     # graphs keep the event
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.flags, cfg.dep = 0, 0
    cfg.comm_kind, cfg.len = 2, 32                                        # own reduce: len must be M*N
    cfg.out = 0x40000
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.len = 64
    expect_accepted(L, L.run_overlap, ctypes.byref(cfg), ctypes.byref(res))  # 8x8 outputs, len 64
    cfg.out = 0x3000 + 2 * 64 * 2 - 8                                     # out inside C_1 (n_iter = 2)
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -4
    cfg.M, cfg.N, cfg.len, cfg.out = 3, 3, 9, 0x40000                     # M*N not a multiple of 8
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.M, cfg.N, cfg.len, cfg.comm_kind, cfg.out = 8, 8, 64, 0, 0x30000
    cfg.N = 12                                                            # K x N needs N % 8 == 0
    assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1
    cfg.gemm_b_layout = 1                                                 # N x K does not
    expect_accepted(L, L.run_overlap, ctypes.byref(cfg), ctypes.byref(res))
    cfg.gemm_b_layout, cfg.N = 0, 8
    for rate in (-1.0, 5.0, float("nan"), 1e7):                          # pacing out of range
        cfg.comm_rate_gbs = rate
        assert L.run_overlap(ctypes.byref(cfg), ctypes.byref(res)) == -1, rate
    assert b.MIN_COMM_RATE_GBS == 10.0
    for rate in (0.0, 10.0, 1500.0):                                      # valid: passes validation
        cfg.comm_rate_gbs = rate
        expect_accepted(L, L.run_overlap, ctypes.byref(cfg), ctypes.byref(res))


def test_gemm_info_argument_errors(L):
    x = ctypes.c_int(0)
    assert L.occ_gemm_info(None, ctypes.byref(x), ctypes.byref(x)) == -1
    assert L.occ_gemm_info(ctypes.byref(x), None, ctypes.byref(x)) == -1
    assert L.occ_gemm_info(ctypes.byref(x), ctypes.byref(x), None) == -1


def test_overlap_tune_argument_errors(L):
    from paper_2606_09200_amd import binding as b
    cfg = b.occ_overlap_cfg()
    res = b.occ_overlap_result()
    pref = ctypes.c_int(0)
    assert L.occ_overlap_tune(None, 2, ctypes.byref(res), ctypes.byref(pref)) == -1
    assert L.occ_overlap_tune(ctypes.byref(cfg), 0, ctypes.byref(res), ctypes.byref(pref)) == -1
    assert L.occ_overlap_tune(ctypes.byref(cfg), 2, None, ctypes.byref(pref)) == -1
    assert L.occ_overlap_tune(ctypes.byref(cfg), 2, ctypes.byref(res), None) == -1
    cfg.n_iter = 0  # invalid schedule: rejected before any device call
    assert L.occ_overlap_tune(ctypes.byref(cfg), 2, ctypes.byref(res), ctypes.byref(pref)) == -1


def test_overlap_enqueue_argument_errors(L):
    from paper_2606_09200_amd import binding as b
    assert L.occ_overlap_workspace_bytes(0) == 0
    assert L.occ_overlap_workspace_bytes(1) == 256
    assert L.occ_overlap_workspace_bytes(10) == 256
    assert L.occ_overlap_workspace_bytes(100) == 1024      # 201 words, rounded up to 256 bytes
    cfg = b.occ_overlap_cfg()
    cfg.M = cfg.N = cfg.K = 8
    cfg.A, cfg.B, cfg.C = 0x1000, 0x2000, 0x3000
    arr = (ctypes.c_void_p * 2)(0x10000, 0x20000)
    cfg.bufs = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    cfg.nchunks, cfg.len, cfg.out, cfg.n_iter = 2, 64, 0x30000, 4
    ws = P(0x50000)
    assert L.occ_overlap_enqueue(None, None, ws, 256, None) == -1
    assert L.occ_overlap_enqueue(ctypes.byref(cfg), None, None, 256, None) == -1     # no workspace
    assert L.occ_overlap_enqueue(ctypes.byref(cfg), None, P(0x50002), 256, None) == -1  # misaligned
    assert L.occ_overlap_enqueue(ctypes.byref(cfg), None, ws, 16, None) == -1       # too short
    cfg.timeline = 0x60000                                                         # no tracing here
    assert L.occ_overlap_enqueue(ctypes.byref(cfg), None, ws, 256, None) == -1
    cfg.timeline = None
    cfg.out = 0x3000 + 16                                                          # output inside C
    assert L.occ_overlap_enqueue(ctypes.byref(cfg), None, ws, 256, None) == -4
    cfg.out = 0x30000
    cfg.reps, cfg.warmup, cfg.flags, cfg.dep = 0, -1, 8, 0                        # fields it does not read
    expect_accepted(L, L.occ_overlap_enqueue, ctypes.byref(cfg), None, ws, 256, None)
    cfg.n_iter = 0
    assert L.occ_overlap_enqueue(ctypes.byref(cfg), None, ws, 256, None) == -1


def test_overlap_enqueue_noalloc_argument_errors(L):
    from paper_2606_09200_amd import binding as b
    assert b.NOALLOC_MAX_ITER == 1024 and "#define OCC_NOALLOC_MAX_ITER 1024" in open(HEADER).read()
    cfg = b.occ_overlap_cfg()
    cfg.M = cfg.N = cfg.K = 8
    cfg.A, cfg.B, cfg.C = 0x1000, 0x2000, 0x3000
    arr = (ctypes.c_void_p * 2)(0x10000, 0x20000)
    cfg.bufs = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
    cfg.nchunks, cfg.len, cfg.out = 2, 64, 0x30000
    assert L.occ_overlap_enqueue_noalloc(None, None, None) == -1
    for n in (0, -3, 1025):                                                       # beyond the array
        cfg.n_iter = n
        assert L.occ_overlap_enqueue_noalloc(ctypes.byref(cfg), None, None) == -1, n
