"""Python binding of libocc.so: the C entry points of include/occ.h, same names.

Argument marshalling only: tensors become device pointers and sizes, the
current torch stream becomes the hipStream_t, a non-zero status becomes an
``OccError``.  Every step of the hot path runs in the library's HIP kernels;
there is no fallback: if libocc.so is missing or no gfx950 GPU is current,
the calls fail loudly.

torch must be imported before the library is loaded so that both use the one
HIP runtime already in the process (torch's; same soname).
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libocc.so")

OCC_OK, OCC_EINVAL, OCC_ELDS, OCC_EPERM, OCC_EALIAS, OCC_EHIP, OCC_ENODEV, OCC_ETIMEOUT = 0, -1, -2, -3, -4, -5, -6, -7
OCC_COMM_REDUCE, OCC_COMM_PERMUTE, OCC_COMM_REDUCE_OWN = 0, 1, 2
OCC_RUN_SEQ, OCC_RUN_OVL, OCC_RUN_ISO, OCC_RUN_GRAPH, OCC_RUN_PACE_ALL = 1, 2, 4, 8, 16
OCC_B_KN, OCC_B_NK = 0, 1
OCC_DEP_EVENT, OCC_DEP_COUNTER = 0, 1
# kernel variants of occ.h, by the layout of B they read
KN_VARIANTS = {
    32: "dl+pipe 256x256x64 8w 2st", 33: "skinny M<=16, 128-column units",
    35: "dl 128x128x64 4w 3st", 36: "opt1 64x64x32 1st", 37: "opt2 64x64x64 1st",
    38: "dl+pipe 128x256x32 4w 2st 2wg/cu", 39: "dl 64x64x64 4w 2st",
}
NK_VARIANTS = {
    6: "opt1 64x64x32 register-staged", 7: "opt2 64x64x64 register-staged", 9: "dl 64x64x64 4w 2st",
    14: "dl 128x128x64 4w 3st", 16: "dl+pipe 256x256x64 8w 2st", 21: "skinny M<=16, 8w, 8 k-blocks in flight",
    25: "dl+pipe 128x256x32 4w 2st 2wg/cu", 34: "skinny M<=16, A in registers, B through LDS (K%1024==0, K<=8192)",
}
SKINNY_VARIANTS = (21, 33, 34)     # M <= 16 only
ABI_VERSION = (2, 2)
NOALLOC_MAX_ITER = 1024   # OCC_NOALLOC_MAX_ITER      # OCC_VERSION_MAJOR, OCC_VERSION_MINOR of the structures below
MIN_COMM_RATE_GBS = 10.0  # OCC_MIN_COMM_RATE_GBS
WG_RECORD_WORDS = 12    # uint32 words per workgroup record in a wg_trace buffer


class OccError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__("%s: %s" % (where, occ_strerror(status)))


class occ_gemm_plan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in (
        "tile_m", "tile_n", "tile_k", "threads", "tile_lds_bytes", "grid", "tiles", "wg_per_cu",
        "max_lds_per_wg", "lds_per_cu", "num_cus", "kernel_id")]


class occ_overlap_cfg(ctypes.Structure):
    _fields_ = [
        ("M", ctypes.c_int), ("N", ctypes.c_int), ("K", ctypes.c_int),
        ("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("C", ctypes.c_void_p),
        ("lds_bytes", ctypes.c_size_t), ("gemm_variant", ctypes.c_int), ("gemm_grid", ctypes.c_int),
        ("gemm_priority", ctypes.c_int), ("gemm_b_layout", ctypes.c_int),
        ("comm_kind", ctypes.c_int), ("bufs", ctypes.POINTER(ctypes.c_void_p)),
        ("nchunks", ctypes.c_int), ("len", ctypes.c_size_t), ("out", ctypes.c_void_p),
        ("src", ctypes.c_void_p), ("dst", ctypes.c_void_p), ("perm", ctypes.POINTER(ctypes.c_int32)),
        ("chunk_bytes", ctypes.c_size_t), ("comm_wgs", ctypes.c_int), ("comm_priority", ctypes.c_int),
        ("comm_rate_gbs", ctypes.c_double),
        ("n_iter", ctypes.c_int), ("dep", ctypes.c_int), ("reps", ctypes.c_int), ("warmup", ctypes.c_int),
        ("flags", ctypes.c_int), ("stream", ctypes.c_void_p), ("timeline", ctypes.c_void_p),
        ("wg_trace", ctypes.c_void_p), ("wg_trace_cap", ctypes.c_int),
    ]


class occ_overlap_result(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in (
        "t_seq_ms", "t_ovl_ms", "t_seq_min_ms", "t_ovl_min_ms", "reduction_pct", "t_gemm_ms",
        "t_comm_ms")] + [(n, ctypes.c_int) for n in (
            "gemm_wg_per_cu", "gemm_grid", "gemm_tile_lds", "comm_wgs")] + [(n, ctypes.c_double) for n in (
                "t_seq_median_ms", "t_ovl_median_ms", "t_seq_std_ms", "t_ovl_std_ms")]


_lib = None
_P = ctypes.c_void_p
_SIGS = {
    "occ_gemm": [_P, _P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_size_t, _P],
    "occ_gemm_ex": [_P, _P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_size_t,
                    ctypes.c_int, ctypes.c_int, _P],
    "occ_gemm_bt": [_P, _P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_size_t, _P],
    "occ_gemm_bt_ex": [_P, _P, _P, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_size_t,
                       ctypes.c_int, ctypes.c_int, _P],
    "occ_gemm_plan_query": [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_size_t, ctypes.c_int,
                            ctypes.c_int, ctypes.POINTER(occ_gemm_plan)],
    "occ_gemm_bt_plan_query": [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_size_t, ctypes.c_int,
                               ctypes.c_int, ctypes.POINTER(occ_gemm_plan)],
    "occ_gemm_info": [ctypes.POINTER(ctypes.c_int)] * 3,
    "share_reduce": [ctypes.POINTER(_P), ctypes.c_int, ctypes.c_size_t, _P, _P],
    "share_reduce_ex": [ctypes.POINTER(_P), ctypes.c_int, ctypes.c_size_t, _P, ctypes.c_int,
                        ctypes.c_int, _P],
    "share_reduce_own": [_P, ctypes.POINTER(_P), ctypes.c_int, ctypes.c_size_t, _P, ctypes.c_int,
                         ctypes.c_int, _P],
    "share_permute": [_P, _P, ctypes.POINTER(ctypes.c_int32), ctypes.c_int, ctypes.c_size_t, _P],
    "share_permute_ex": [_P, _P, ctypes.POINTER(ctypes.c_int32), ctypes.c_int, ctypes.c_size_t,
                         ctypes.c_int, ctypes.c_int, _P],
    "run_overlap": [ctypes.POINTER(occ_overlap_cfg), ctypes.POINTER(occ_overlap_result)],
    "occ_overlap_tune": [ctypes.POINTER(occ_overlap_cfg), ctypes.c_int,
                         ctypes.POINTER(occ_overlap_result), ctypes.POINTER(ctypes.c_int)],
    "occ_overlap_workspace_bytes": [ctypes.c_int],
    "occ_overlap_enqueue": [ctypes.POINTER(occ_overlap_cfg), _P, _P, ctypes.c_size_t, _P],
    "occ_overlap_enqueue_noalloc": [ctypes.POINTER(occ_overlap_cfg), _P, _P],
    "occ_strerror": [ctypes.c_int],
    "occ_version": [],
}


def lib():
    """The loaded libocc.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libocc.so is not built (%s); run python -m paper_2606_09200_amd.build"
                               % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = (ctypes.c_char_p if name == "occ_strerror" else
                         ctypes.c_size_t if name == "occ_overlap_workspace_bytes" else ctypes.c_int)
        v = L.occ_version()
        if (v >> 16, v & 0xFFFF) != ABI_VERSION:
            raise RuntimeError("%s has ABI version %d.%d, this binding expects %d.%d; rebuild it with "
                               "python -m paper_2606_09200_amd.build" % ((LIB_PATH, v >> 16, v & 0xFFFF) + ABI_VERSION))
        _lib = L
    return _lib


def occ_strerror(status):
    return lib().occ_strerror(int(status)).decode()


def occ_version():
    v = lib().occ_version()
    return (v >> 16, v & 0xFFFF)


def _check(status, where):
    if status != OCC_OK:
        raise OccError(status, where)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else ctypes.c_void_p(0)


def _gemm_args(A, B, C, b_kn=True):
    for name, t in (("A", A), ("B", B), ("C", C)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or t.dim() != 2:
            raise ValueError("%s must be a contiguous 2-D bfloat16 GPU tensor" % name)
    M, K = A.shape
    N = B.shape[1] if b_kn else B.shape[0]
    if B.shape[0 if b_kn else 1] != K or tuple(C.shape) != (M, N):
        raise ValueError("shapes must be A (M,K), B (%s), C (M,N)" % ("K,N" if b_kn else "N,K"))
    return M, N, K


def occ_gemm(A, B, C, lds_bytes=0, stream=None):
    """C = A @ B (bf16, fp32 accumulation); B is K x N."""
    M, N, K = _gemm_args(A, B, C)
    _check(lib().occ_gemm(_ptr(A), _ptr(B), _ptr(C), M, N, K, int(lds_bytes), _stream(stream)),
           "occ_gemm")
    return C


def occ_gemm_ex(A, B, C, lds_bytes=0, variant=0, grid_cap=0, stream=None):
    """occ_gemm with a K x N kernel variant and a persistent grid cap."""
    M, N, K = _gemm_args(A, B, C)
    _check(lib().occ_gemm_ex(_ptr(A), _ptr(B), _ptr(C), M, N, K, int(lds_bytes), int(variant),
                             int(grid_cap), _stream(stream)), "occ_gemm_ex")
    return C


def occ_gemm_bt(A, B, C, lds_bytes=0, stream=None):
    """C = A @ B.T (bf16, fp32 accumulation); B is N x K (a linear layer's weight)."""
    M, N, K = _gemm_args(A, B, C, b_kn=False)
    _check(lib().occ_gemm_bt(_ptr(A), _ptr(B), _ptr(C), M, N, K, int(lds_bytes), _stream(stream)),
           "occ_gemm_bt")
    return C


def occ_gemm_bt_ex(A, B, C, lds_bytes=0, variant=0, grid_cap=0, stream=None):
    """occ_gemm_bt with an N x K kernel variant and a persistent grid cap."""
    M, N, K = _gemm_args(A, B, C, b_kn=False)
    _check(lib().occ_gemm_bt_ex(_ptr(A), _ptr(B), _ptr(C), M, N, K, int(lds_bytes), int(variant),
                                int(grid_cap), _stream(stream)), "occ_gemm_bt_ex")
    return C


def occ_gemm_plan_query(M, N, K, lds_bytes=0, variant=0, grid_cap=0, strict=False, b_layout="kn"):
    """Plan as a dict; 'feasible' is False when the pad does not fit (OCC_ELDS).
    b_layout "kn" (default) is occ_gemm's plan, "nk" occ_gemm_bt's."""
    if b_layout not in ("nk", "kn"):
        raise ValueError("b_layout must be 'kn' or 'nk'")
    name = "occ_gemm_plan_query" if b_layout == "kn" else "occ_gemm_bt_plan_query"
    p = occ_gemm_plan()
    st = getattr(lib(), name)(int(M), int(N), int(K), int(lds_bytes), int(variant), int(grid_cap),
                              ctypes.byref(p))
    if st not in (OCC_OK, OCC_ELDS) or (strict and st != OCC_OK):
        raise OccError(st, name)
    d = {f: getattr(p, f) for f, _ in occ_gemm_plan._fields_}
    d["feasible"] = st == OCC_OK
    return d


def occ_gemm_bt_plan_query(M, N, K, lds_bytes=0, variant=0, grid_cap=0, strict=False):
    """occ_gemm_bt's plan (B stored N x K) as a dict, as occ_gemm_plan_query."""
    return occ_gemm_plan_query(M, N, K, lds_bytes, variant, grid_cap, strict, b_layout="nk")


def occ_gemm_info():
    """(S_tile of the large-shape kernel, max LDS per workgroup, LDS per CU), bytes."""
    v = [ctypes.c_int(0) for _ in range(3)]
    _check(lib().occ_gemm_info(*[ctypes.byref(x) for x in v]), "occ_gemm_info")
    return tuple(x.value for x in v)


def _chunk_ptrs(bufs):
    if isinstance(bufs, torch.Tensor):
        bufs = list(bufs.unbind(0)) if bufs.dim() == 2 else [bufs]
    for b in bufs:
        if b.dtype != torch.float32 or not b.is_cuda or not b.is_contiguous():
            raise ValueError("chunks must be contiguous float32 GPU tensors")
    length = bufs[0].numel() if bufs else 0
    if any(b.numel() != length for b in bufs):
        raise ValueError("all chunks must have the same length")
    arr = (ctypes.c_void_p * max(1, len(bufs)))(*[b.data_ptr() for b in bufs])
    return arr, len(bufs), length


def share_reduce(bufs, out, stream=None, wgs=0, priority=0):
    """out = bufs[0] + bufs[1] + ... (binary32, left to right)."""
    arr, n, length = _chunk_ptrs(bufs)
    if out.dtype != torch.float32 or not out.is_cuda or out.numel() != length:
        raise ValueError("out must be a float32 GPU tensor of the chunk length")
    if wgs or priority:
        st = lib().share_reduce_ex(arr, n, length, _ptr(out), int(wgs), int(priority), _stream(stream))
    else:
        st = lib().share_reduce(arr, n, length, _ptr(out), _stream(stream))
    _check(st, "share_reduce")
    return out


def _peer_ptrs(peers, length):
    """Host array of fp32 peer-chunk pointers (possibly none) of `length` elements each."""
    if peers is None:
        peers = []
    elif isinstance(peers, torch.Tensor):
        peers = list(peers.unbind(0)) if peers.dim() == 2 else [peers]
    for b in peers:
        if b.dtype != torch.float32 or not b.is_cuda or not b.is_contiguous() or b.numel() != length:
            raise ValueError("peer chunks must be contiguous float32 GPU tensors of the own length")
    arr = (ctypes.c_void_p * max(1, len(peers)))(*[b.data_ptr() for b in peers])
    return arr, len(peers)


def share_reduce_own(own, peers, out, stream=None, wgs=0, priority=0):
    """out = f32(own) + peers[0] + peers[1] + ... (binary32, left to right); own is bf16."""
    if own.dtype != torch.bfloat16 or not own.is_cuda or not own.is_contiguous():
        raise ValueError("own must be a contiguous bfloat16 GPU tensor")
    length = own.numel()
    arr, n = _peer_ptrs(peers, length)
    if out.dtype != torch.float32 or not out.is_cuda or out.numel() != length:
        raise ValueError("out must be a float32 GPU tensor of the own length")
    _check(lib().share_reduce_own(_ptr(own), arr, n, length, _ptr(out), int(wgs), int(priority),
                                  _stream(stream)), "share_reduce_own")
    return out


def _perm_arr(perm):
    p = [int(x) for x in (perm.tolist() if hasattr(perm, "tolist") else perm)]
    return (ctypes.c_int32 * max(1, len(p)))(*p), len(p)


def share_permute(src, dst, perm, chunk_bytes, stream=None, wgs=0, priority=0):
    """dst chunk i = src chunk perm[i] (byte copy)."""
    arr, n = _perm_arr(perm)
    for name, t in (("src", src), ("dst", dst)):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("%s must be a contiguous GPU tensor" % name)
        if t.numel() * t.element_size() != n * chunk_bytes:
            raise ValueError("%s must hold nchunks * chunk_bytes bytes" % name)
    if wgs or priority:
        st = lib().share_permute_ex(_ptr(src), _ptr(dst), arr, n, int(chunk_bytes), int(wgs),
                                    int(priority), _stream(stream))
    else:
        st = lib().share_permute(_ptr(src), _ptr(dst), arr, n, int(chunk_bytes), _stream(stream))
    _check(st, "share_permute")
    return dst


def decode_wg_trace(wg_trace):
    """Records of a filled wg_trace tensor as a list of dicts (host side)."""
    w = wg_trace.cpu().numpy().astype("int64") & 0xFFFFFFFF
    n = min(int(w[0]), (w.size - 4) // WG_RECORD_WORDS)
    out = []
    for i in range(n):
        r = w[4 + WG_RECORD_WORDS * i: 4 + WG_RECORD_WORDS * (i + 1)]
        hw, xcc = int(r[2]), int(r[3])
        out.append({"tag": int(r[0]), "iter": int(r[0]) >> 1, "kind": "comm" if r[0] & 1 else "gemm",
                    "block": int(r[1]), "cu": (hw >> 8) & 0xF, "sh": (hw >> 12) & 1,
                    "se": (hw >> 13) & 0x7, "xcc": xcc & 0xF,
                    "t0": int(r[4]) | (int(r[5]) << 32), "t1": int(r[6]) | (int(r[7]) << 32),
                    "cycles": int(r[8]) | (int(r[9]) << 32)})
    return out


def _make_cfg(A, B, C, bufs, out, src, dst, perm, chunk_bytes, lds_bytes, gemm_variant, gemm_grid,
              gemm_priority, comm_wgs, comm_priority, n_iter, reps, warmup, flags, timeline, wg_trace,
              comm_rate_gbs=0.0, b_layout="kn", reduce_own=False, dep="event", stream=None):
    if b_layout not in ("nk", "kn"):
        raise ValueError("b_layout must be 'kn' or 'nk'")
    if dep not in ("event", "counter"):
        raise ValueError("dep must be 'event' or 'counter'")
    if reduce_own:
        # C holds one M x N output per iteration; the collective reduces its own
        if C.dim() != 3 or C.shape[0] != n_iter:
            raise ValueError("with reduce_own, C must be (n_iter, M, N)")
        M, N, K = _gemm_args(A, B, C[0], b_kn=b_layout == "kn")
    else:
        M, N, K = _gemm_args(A, B, C, b_kn=b_layout == "kn")
    cfg = occ_overlap_cfg()
    cfg.M, cfg.N, cfg.K = M, N, K
    cfg.A, cfg.B, cfg.C = _ptr(A).value, _ptr(B).value, _ptr(C).value
    cfg.lds_bytes, cfg.gemm_variant, cfg.gemm_grid = int(lds_bytes), int(gemm_variant), int(gemm_grid)
    cfg.gemm_priority = int(gemm_priority)
    cfg.comm_rate_gbs = float(comm_rate_gbs)
    cfg.gemm_b_layout = OCC_B_KN if b_layout == "kn" else OCC_B_NK
    cfg.dep = OCC_DEP_COUNTER if dep == "counter" else OCC_DEP_EVENT
    cfg.stream = _stream(stream).value
    keep = []
    if reduce_own:
        arr, n = _peer_ptrs(bufs, M * N)
        keep.append(arr)
        cfg.comm_kind = OCC_COMM_REDUCE_OWN
        cfg.bufs = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
        cfg.nchunks, cfg.len, cfg.out = n, M * N, _ptr(out).value
        if out.numel() != M * N or out.dtype != torch.float32:
            raise ValueError("out must be float32 of M*N elements")
    elif bufs is not None:
        arr, n, length = _chunk_ptrs(bufs)
        keep.append(arr)
        cfg.comm_kind = OCC_COMM_REDUCE
        cfg.bufs = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
        cfg.nchunks, cfg.len, cfg.out = n, length, _ptr(out).value
        if out.numel() != length or out.dtype != torch.float32:
            raise ValueError("out must be float32 of the chunk length")
    else:
        parr, n = _perm_arr(perm)
        keep.append(parr)
        cfg.comm_kind = OCC_COMM_PERMUTE
        cfg.src, cfg.dst = _ptr(src).value, _ptr(dst).value
        cfg.perm = ctypes.cast(parr, ctypes.POINTER(ctypes.c_int32))
        cfg.nchunks, cfg.chunk_bytes = n, int(chunk_bytes)
        for t in (src, dst):
            if t.numel() * t.element_size() != n * chunk_bytes:
                raise ValueError("src/dst must hold nchunks * chunk_bytes bytes")
    cfg.comm_wgs, cfg.comm_priority = int(comm_wgs), int(comm_priority)
    cfg.n_iter, cfg.reps, cfg.warmup, cfg.flags = int(n_iter), int(reps), int(warmup), int(flags)
    if timeline is not None:
        if timeline.dtype not in (torch.int64, torch.uint64) or timeline.numel() < 4 * n_iter:
            raise ValueError("timeline must hold 4*n_iter 64-bit entries")
        cfg.timeline = timeline.data_ptr()
    if wg_trace is not None:
        if wg_trace.dtype not in (torch.int32, torch.uint32) or wg_trace.numel() < 4 + WG_RECORD_WORDS:
            raise ValueError("wg_trace must be a 32-bit tensor of 4 + %d*cap entries" % WG_RECORD_WORDS)
        cfg.wg_trace = wg_trace.data_ptr()
        cfg.wg_trace_cap = (wg_trace.numel() - 4) // WG_RECORD_WORDS
    return cfg, keep


def run_overlap(A, B, C, *, bufs=None, out=None, src=None, dst=None, perm=None, chunk_bytes=0,
                lds_bytes=0, gemm_variant=0, gemm_grid=0, gemm_priority=0, comm_wgs=0,
                comm_priority=3, n_iter=10, reps=20, warmup=10, flags=0, timeline=None,
                wg_trace=None, comm_rate_gbs=0.0, b_layout="kn", reduce_own=False, dep="event",
                stream=None):
    """Sequential vs overlapped makespan of n_iter GEMM -> collective iterations.

    Pass ``bufs``/``out`` for the allreduce share, or ``src``/``dst``/``perm``/
    ``chunk_bytes`` for the alltoall share.  ``timeline``: optional uint64 GPU
    tensor of 4*n_iter entries (see occ_overlap_cfg.timeline).  ``wg_trace``:
    optional int32 GPU tensor of 4 + 12*cap entries (see occ_overlap_cfg.wg_trace).
    ``comm_rate_gbs``: bandwidth pacing of the collective in the overlapped
    schedule (0 = full speed).  ``b_layout``: "kn" (B is K x N, C = A B, the
    default) or "nk" (B is N x K, C = A B^T).  ``reduce_own``: the collective
    consumes the GEMM's output (OCC_COMM_REDUCE_OWN): C is (n_iter, M, N),
    iteration i's GEMM writes C[i] and its collective is
    share_reduce_own(C[i], bufs, out) with ``bufs`` the fp32 peer chunks
    (possibly none).  ``dep``: the per-iteration dependency, "event" or
    "counter" (OCC_DEP_COUNTER).  The library's streams start after the work
    already queued on ``stream`` (default: torch's current stream).  Returns
    the occ_overlap_result fields as a dict.
    """
    cfg, keep = _make_cfg(A, B, C, bufs, out, src, dst, perm, chunk_bytes, lds_bytes, gemm_variant,
                          gemm_grid, gemm_priority, comm_wgs, comm_priority, n_iter, reps, warmup,
                          flags, timeline, wg_trace, comm_rate_gbs, b_layout, reduce_own, dep, stream)
    res = occ_overlap_result()
    _check(lib().run_overlap(ctypes.byref(cfg), ctypes.byref(res)), "run_overlap")
    return {f: getattr(res, f) for f, _ in occ_overlap_result._fields_}


def occ_overlap_tune(A, B, C, *, bufs=None, out=None, src=None, dst=None, perm=None, chunk_bytes=0,
                     gemm_variant=0, n_iter=10, reps=20, warmup=10, tune_reps=3, b_layout="kn",
                     reduce_own=False, stream=None):
    """Adaptive knob choice (see occ.h).  Returns (chosen knobs, result dict, prefer_sequential)."""
    cfg, keep = _make_cfg(A, B, C, bufs, out, src, dst, perm, chunk_bytes, 0, gemm_variant, 0, 0, 0,
                          0, n_iter, reps, warmup, 0, None, None, 0.0, b_layout, reduce_own, "event", stream)
    res = occ_overlap_result()
    pref = ctypes.c_int(0)
    _check(lib().occ_overlap_tune(ctypes.byref(cfg), int(tune_reps), ctypes.byref(res),
                                  ctypes.byref(pref)), "occ_overlap_tune")
    knobs = {"comm_priority": cfg.comm_priority, "comm_wgs": cfg.comm_wgs,
             "gemm_grid": cfg.gemm_grid, "lds_bytes": cfg.lds_bytes,
             "dep": "counter" if cfg.dep == OCC_DEP_COUNTER else "event"}
    return knobs, {f: getattr(res, f) for f, _ in occ_overlap_result._fields_}, bool(pref.value)


def occ_overlap_workspace_bytes(n_iter):
    """Device bytes occ_overlap_enqueue needs for n_iter iterations."""
    return int(lib().occ_overlap_workspace_bytes(int(n_iter)))


def occ_overlap_enqueue(A, B, C, *, workspace, comm_stream, err=None, bufs=None, out=None, src=None, dst=None,
                        perm=None, chunk_bytes=0, lds_bytes=0, gemm_variant=0, gemm_grid=0, gemm_priority=0,
                        comm_wgs=0, comm_priority=0, n_iter=10, comm_rate_gbs=0.0, b_layout="kn",
                        reduce_own=False, stream=None):
    """Enqueue the overlapped schedule (GEMMs on ``stream``, default torch's
    current stream; collectives on ``comm_stream``) with the device-counter
    dependency in ``workspace`` (a zeroed GPU tensor of at least
    occ_overlap_workspace_bytes(n_iter) bytes) and return; ``err``: optional
    int32 GPU tensor of one element set to 1 if a bounded wait ran out."""
    cfg, keep = _make_cfg(A, B, C, bufs, out, src, dst, perm, chunk_bytes, lds_bytes, gemm_variant,
                          gemm_grid, gemm_priority, comm_wgs, comm_priority, n_iter, 1, 0, 0, None, None,
                          comm_rate_gbs, b_layout, reduce_own, "counter", stream)
    if not workspace.is_cuda or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous GPU tensor")
    if err is not None and (not err.is_cuda or err.element_size() != 4 or err.numel() < 1):
        raise ValueError("err must be a 32-bit GPU tensor")
    _check(lib().occ_overlap_enqueue(ctypes.byref(cfg), _stream(comm_stream), _ptr(workspace),
                                     workspace.numel() * workspace.element_size(), _ptr(err)),
           "occ_overlap_enqueue")


def occ_overlap_enqueue_noalloc(A, B, C, *, comm_stream, err=None, bufs=None, out=None, src=None, dst=None,
                                perm=None, chunk_bytes=0, lds_bytes=0, gemm_variant=0, gemm_grid=0,
                                gemm_priority=0, comm_wgs=0, comm_priority=0, n_iter=10, comm_rate_gbs=0.0,
                                b_layout="kn", reduce_own=False, stream=None):
    """occ_overlap_enqueue with the counters in the library's own static
    device array (at most NOALLOC_MAX_ITER iterations): allocates nothing."""
    cfg, keep = _make_cfg(A, B, C, bufs, out, src, dst, perm, chunk_bytes, lds_bytes, gemm_variant,
                          gemm_grid, gemm_priority, comm_wgs, comm_priority, n_iter, 1, 0, 0, None, None,
                          comm_rate_gbs, b_layout, reduce_own, "counter", stream)
    if err is not None and (not err.is_cuda or err.element_size() != 4 or err.numel() < 1):
        raise ValueError("err must be a 32-bit GPU tensor")
    _check(lib().occ_overlap_enqueue_noalloc(ctypes.byref(cfg), _stream(comm_stream), _ptr(err)),
           "occ_overlap_enqueue_noalloc")
