"""CPU oracle for the GEMM + communication-share hot path.

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product library
never calls it and shares no code with it; the two meet only in the seeded
input generators, which hold none of the method's arithmetic.

What each function computes (the plain definitions, see ``oracle.c``):

* :func:`gemm_bf16` -- Background, item 1 (the GEMM ``C = alpha op(A) op(B) +
  beta C``), read with alpha = 1, beta = 0: the products accumulated in
  binary32 in increasing k (``acc="f32"``, the workload's definition) or
  summed exactly in binary64 (``acc="f64"``), then one round-to-nearest-even
  to bfloat16.
* :func:`chunk_sum_f32` -- Background, item 2 (allreduce aggregates local
  gradients): one GPU's share is the element-wise binary32 sum of its chunks
  in the fixed order ``c0 + c1 + ... + c_{n-1}``.
* :func:`permute_chunks` -- Background, item 2 (alltoall routes tokens between
  devices): chunk ``i`` of the output is chunk ``perm[i]`` of the input.
* :mod:`oracle.schedule` -- Section 3.2-3.3 (per-iteration dependency
  ``K_g^i -> K_c^i``) and Section 4.2 (TimeRatio, overlap rate).
"""
import ctypes

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(_build.ensure_built())
        lib.oracle_gemm_bf16_block.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
            ctypes.c_void_p]
        lib.oracle_gemm_bf16_block.restype = None
        lib.oracle_gemm_bf16_f32acc_block.argtypes = lib.oracle_gemm_bf16_block.argtypes
        lib.oracle_gemm_bf16_f32acc_block.restype = None
        lib.oracle_chunk_sum_f32.argtypes = [
            ctypes.POINTER(ctypes.c_void_p), ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p]
        lib.oracle_chunk_sum_f32.restype = None
        lib.oracle_chunk_sum_own_f32.argtypes = [
            ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p), ctypes.c_int, ctypes.c_size_t,
            ctypes.c_void_p]
        lib.oracle_chunk_sum_own_f32.restype = None
        lib.oracle_permute.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t]
        lib.oracle_permute.restype = None
        lib.oracle_double_to_bf16.argtypes = [ctypes.c_double]
        lib.oracle_double_to_bf16.restype = ctypes.c_uint16
        lib.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        lib.oracle_bf16_to_double.restype = ctypes.c_double
        lib.oracle_num_threads.argtypes = []
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops run on in this process."""
    return int(_load().oracle_num_threads())


def _u16(x):
    """View a bfloat16 tensor / uint16 array as a C-contiguous numpy uint16 array."""
    if hasattr(x, "view") and hasattr(x, "numpy") and not isinstance(x, np.ndarray):
        import torch
        if x.dtype == torch.bfloat16:
            x = x.view(torch.int16)
        x = x.contiguous().numpy()
    x = np.ascontiguousarray(x)
    if x.dtype.itemsize != 2:
        raise TypeError("expected 16-bit bfloat16 bit patterns, got %s" % x.dtype)
    return x.view(np.uint16)


def double_to_bf16(x: float) -> int:
    """bfloat16 bit pattern of ``x`` rounded once, to nearest, ties to even."""
    return int(_load().oracle_double_to_bf16(float(x)))


def bf16_to_double(h: int) -> float:
    return float(_load().oracle_bf16_to_double(int(h) & 0xFFFF))


def gemm_bf16(A, B, M, N, K, b_layout="nk", rows=None, cols=None, acc="f32"):
    """bf16 bit patterns of ``C = A @ op(B)``, or of its block ``C[rows, cols]``.

    ``A`` is M x K row-major.  ``b_layout="nk"``: ``B`` is stored N x K (a linear
    layer's weight, op(B) = B^T); ``"kn"``: ``B`` is stored K x N.
    ``rows``/``cols`` are half-open ``(start, stop)`` ranges (default: all).
    ``acc="f32"``: binary32 accumulation in increasing k; ``"f64"``: the exact
    sum.  Returns a numpy uint16 array of shape (rows, cols).
    """
    a = _u16(A).reshape(-1)
    b = _u16(B).reshape(-1)
    if a.size != M * K or b.size != N * K:
        raise ValueError("operand sizes do not match M, N, K")
    m0, m1 = rows if rows is not None else (0, M)
    n0, n1 = cols if cols is not None else (0, N)
    if not (0 <= m0 <= m1 <= M and 0 <= n0 <= n1 <= N):
        raise ValueError("block out of range")
    out = np.empty((m1 - m0, n1 - n0), dtype=np.uint16)
    lay = {"nk": 0, "kn": 1}[b_layout]
    fn = {"f32": _load().oracle_gemm_bf16_f32acc_block, "f64": _load().oracle_gemm_bf16_block}[acc]
    fn(a.ctypes.data, b.ctypes.data, M, N, K, lay, m0, m1, n0, n1, out.ctypes.data)
    return out


def chunk_sum_f32(chunks):
    """Fixed-order binary32 sum of the rows of ``chunks`` (nchunks x len)."""
    c = np.ascontiguousarray(np.asarray(chunks, dtype=np.float32))
    if c.ndim != 2 or c.shape[0] < 1:
        raise ValueError("chunks must be a non-empty 2-D array")
    n, length = c.shape
    out = np.empty(length, dtype=np.float32)
    ptrs = (ctypes.c_void_p * n)(*[c[i].ctypes.data for i in range(n)])
    _load().oracle_chunk_sum_f32(ptrs, n, length, out.ctypes.data)
    return out


def chunk_sum_own_f32(own, chunks):
    """Fixed-order binary32 sum own + chunks[0] + ... + chunks[n-1], where
    ``own`` holds bfloat16 bit patterns (uint16, or a bfloat16 tensor) of the
    chunk length and ``chunks`` is n x len float32 (n may be 0)."""
    o = np.ascontiguousarray(_u16(own).reshape(-1))
    c = np.ascontiguousarray(np.asarray(chunks, dtype=np.float32)).reshape(-1, o.size)
    n, length = c.shape
    out = np.empty(length, dtype=np.float32)
    ptrs = (ctypes.c_void_p * max(1, n))(*[c[i].ctypes.data for i in range(n)])
    _load().oracle_chunk_sum_own_f32(o.ctypes.data, ptrs, n, length, out.ctypes.data)
    return out


def permute_chunks(src, perm, chunk_bytes):
    """Byte array whose chunk ``i`` is chunk ``perm[i]`` of ``src``."""
    s = np.ascontiguousarray(src).reshape(-1).view(np.uint8)
    p = np.ascontiguousarray(np.asarray(perm, dtype=np.int32))
    n = p.size
    if s.size != n * chunk_bytes:
        raise ValueError("src size must be nchunks * chunk_bytes")
    if sorted(p.tolist()) != list(range(n)):
        raise ValueError("perm is not a permutation of range(nchunks)")
    out = np.empty(n * chunk_bytes, dtype=np.uint8)
    _load().oracle_permute(s.ctypes.data, out.ctypes.data, p.ctypes.data, n, chunk_bytes)
    return out
