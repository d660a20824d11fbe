"""fp64 CPU oracle for the dense contraction (matmul, conv2d).

TEST INFRASTRUCTURE ONLY: imported by the tests, by the smoke check and by the
benchmark's CPU-baseline leg, never by the product path.  It wraps
``liboracle.so`` (built from ``oracle.c`` by ``oracle/build.py``) with numpy
marshalling and shares no code with the HIP library.

Definitions (paper, Sec. 3.1 and Fig. 2; conv2d read as zero-padded
cross-correlation, NCHW / OIHW):

* ``matmul``: ``C[i,j] = sum_k A[i,k] * B[k,j]``, fp64, ascending k.
* ``conv2d``: ``Y[n,oc,oh,ow] = sum_{ic,kh,kw} X[n,ic,oh*s-p+kh,ow*s-p+kw] *
  W[oc,ic,kh,kw]`` with out-of-range input terms zero, fp64, ascending
  (ic, kh, kw).
* ``relu``: elementwise ``v < 0 ? 0 : v`` (one of the paper's operators,
  Sec. 3.1; the consumer of the matmul in its matmul+relu graph, Fig. 9).  A
  NaN stays NaN.  The fused forms are ``relu(matmul(A, B))`` and
  ``relu(conv2d(X, W))``: the consumer applied to the finished fp64 result.

Operands are fp32 arrays, or uint16 arrays holding bf16 bit patterns (widened
exactly).  Both operands of one call must be of the same kind.

The comparison metric used against the GPU (relative Frobenius error) is also
here, as :func:`rel_fro`.
"""
from __future__ import annotations

import ctypes
import os
import time

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_i64 = ctypes.c_int64
_vp = ctypes.c_void_p
_int = ctypes.c_int


def _load(path: str | None = None):
    """Load (and cache) the oracle library; build it if absent."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from oracle import build as _b
            _b.build()
        _lib = _bind(ctypes.CDLL(_LIB_PATH))
    return _lib


def _bind(lib):
    lib.xo_matmul_rows.argtypes = [_i64, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _i64,
                                   _int, _i64, _i64, _int]
    lib.xo_matmul_rows.restype = _int
    lib.xo_matmul_sampled.argtypes = [_i64, _i64, _i64, _vp, _i64, _vp, _i64, _int,
                                      _vp, _vp, _i64, _vp, _int]
    lib.xo_matmul_sampled.restype = None
    lib.xo_conv2d_full.argtypes = [_i64] * 11 + [_vp, _vp, _int, _vp, _int]
    lib.xo_conv2d_full.restype = None
    lib.xo_conv2d_sampled.argtypes = [_i64] * 11 + [_vp, _vp, _int, _vp, _i64, _vp, _int]
    lib.xo_conv2d_sampled.restype = None
    lib.xo_max_threads.argtypes = []
    lib.xo_max_threads.restype = _int
    return lib


def _kind(*arrs) -> int:
    kinds = set()
    for a in arrs:
        if a.dtype == np.float32:
            kinds.add(0)
        elif a.dtype == np.uint16:
            kinds.add(1)
        else:
            raise TypeError("oracle operands must be float32 or uint16 (bf16 bits), got %s" % a.dtype)
    if len(kinds) != 1:
        raise TypeError("oracle operands must all be fp32 or all bf16")
    return kinds.pop()


def _c(a):
    return np.ascontiguousarray(a)


def _ptr(a):
    return a.ctypes.data_as(_vp)


def max_threads(lib=None) -> int:
    return (lib or _load()).xo_max_threads()


def matmul(A: np.ndarray, B: np.ndarray, rows=None, nthreads: int = 0, lib=None) -> np.ndarray:
    """Full fp64 product ``A @ B`` (or rows ``rows=(r0, r1)`` of it, returned
    as an ``(r1 - r0, N)`` array)."""
    lib = lib or _load()
    A, B = _c(A), _c(B)
    M, K = A.shape
    K2, N = B.shape
    if K2 != K:
        raise ValueError("inner dimensions differ")
    r0, r1 = (0, M) if rows is None else rows
    C = np.zeros((M, N), dtype=np.float64) if rows is None else np.zeros((r1 - r0, N), np.float64)
    # For a row slab, offset the A pointer so that row r0 lands at C row 0.
    a_off = A[r0:] if rows is not None else A
    rc = lib.xo_matmul_rows(r1 - r0, N, K, _ptr(_c(a_off)), K, _ptr(B), N, _ptr(C), N,
                            _kind(A, B), 0, r1 - r0, nthreads)
    if rc != 0:
        raise MemoryError("oracle matmul: allocation failed")
    return C


def matmul_sampled(A, B, I, J, nthreads: int = 0, lib=None) -> np.ndarray:
    """fp64 ``(A @ B)[I[s], J[s]]`` for every s."""
    lib = lib or _load()
    A, B = _c(A), _c(B)
    M, K = A.shape
    _, N = B.shape
    I = np.ascontiguousarray(I, dtype=np.int64)
    J = np.ascontiguousarray(J, dtype=np.int64)
    out = np.zeros(I.shape[0], dtype=np.float64)
    lib.xo_matmul_sampled(M, N, K, _ptr(A), K, _ptr(B), N, _kind(A, B), _ptr(I), _ptr(J),
                          I.shape[0], _ptr(out), nthreads)
    return out


def conv2d(X, W, stride=1, pad=0, nthreads: int = 0, lib=None) -> np.ndarray:
    """Full fp64 direct convolution, NCHW x OIHW -> NCHW."""
    lib = lib or _load()
    X, W = _c(X), _c(W)
    N, C, H, Wd = X.shape
    OC, C2, R, S = W.shape
    if C2 != C:
        raise ValueError("channel counts differ")
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    OH = (H + 2 * ph - R) // sh + 1
    OW = (Wd + 2 * pw - S) // sw + 1
    Y = np.zeros((N, OC, max(OH, 0), max(OW, 0)), dtype=np.float64)
    lib.xo_conv2d_full(N, C, H, Wd, OC, R, S, sh, sw, ph, pw, _ptr(X), _ptr(W),
                       _kind(X, W), _ptr(Y), nthreads)
    return Y


def conv2d_sampled(X, W, F, stride=1, pad=0, nthreads: int = 0, lib=None) -> np.ndarray:
    """fp64 conv outputs at flat NCHW indices ``F``."""
    lib = lib or _load()
    X, W = _c(X), _c(W)
    N, C, H, Wd = X.shape
    OC, _, R, S = W.shape
    sh, sw = (stride, stride) if np.isscalar(stride) else stride
    ph, pw = (pad, pad) if np.isscalar(pad) else pad
    F = np.ascontiguousarray(F, dtype=np.int64)
    out = np.zeros(F.shape[0], dtype=np.float64)
    lib.xo_conv2d_sampled(N, C, H, Wd, OC, R, S, sh, sw, ph, pw, _ptr(X), _ptr(W),
                          _kind(X, W), _ptr(F), F.shape[0], _ptr(out), nthreads)
    return out


def relu(v) -> np.ndarray:
    """Elementwise ``v < 0 ? 0 : v`` in fp64 (NaN propagates)."""
    v = np.asarray(v, dtype=np.float64)
    return np.where(v < 0.0, 0.0, v)


def rel_fro(got, ref) -> float:
    """Relative Frobenius error ``||got - ref||_F / ||ref||_F`` (computed in
    fp64).  When ``ref`` is all zero, returns 0.0 if ``got`` is all zero too
    and ``inf`` otherwise."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((got - ref).ravel())
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return float(num / den)


def timed(fn, *args, **kw):
    """(result, seconds) of one call, on a monotonic clock."""
    t0 = time.perf_counter()
    r = fn(*args, **kw)
    return r, time.perf_counter() - t0
