"""Python binding of ``libxtc.so``, the MI355X (gfx950) tiled dense contraction.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``libxtc.so``.  The functions ``xtc_matmul``, ``xtc_conv2d_nchw``,
``xtc_matmul_relu``, ``xtc_conv2d_nchw_relu``, ``xtc_default_schedule``, ``xtc_sched_check``, ``xtc_sched_list``,
``xtc_status_str`` mirror the C ABI of ``include/xtc.h`` one to one (pointers
are Python ints holding device addresses; the stream is a ``hipStream_t`` as
an int, 0 for the null stream).  ``matmul`` and ``conv2d_nchw`` are
conveniences over torch device tensors (torch provides memory and the
current stream, nothing else).

If the library has not been built, importing this package raises
``ImportError``: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libxtc.so")

XTC_F32 = 0
XTC_BF16 = 1
XTC_OP_MATMUL = 0
XTC_OP_CONV2D = 1

XTC_OK = 0
XTC_ERR_NULL_POINTER = 1
XTC_ERR_BAD_SHAPE = 2
XTC_ERR_BAD_LEADING_DIM = 3
XTC_ERR_BAD_DTYPE = 4
XTC_ERR_BAD_SCHEDULE = 5
XTC_ERR_UNSUPPORTED_SCHEDULE = 6
XTC_ERR_TOO_LARGE = 7
XTC_ERR_HIP = 8
XTC_ERR_MISALIGNED = 9


class Sched(ctypes.Structure):
    """``xtc_sched``: see include/xtc.h for the meaning of each field."""
    _fields_ = [(n, ctypes.c_int32) for n in (
        "size", "block_m", "block_n", "block_k", "wave_m", "wave_n",
        "mfma_m", "mfma_n", "mfma_k", "lds_stages", "lds_pad", "unroll_k",
        "raster", "xcd_remap", "k_order", "k_split")]

    def __init__(self, **kw):
        super().__init__()
        self.size = ctypes.sizeof(Sched)
        self.k_split = 1
        for k, v in kw.items():
            setattr(self, k, v)

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_ if n != "size"}

    def __repr__(self):
        d = self.as_dict()
        return ("Sched(block=%dx%dx%d wave=%dx%d mfma=%dx%dx%d stages=%d pad=%d unroll=%d "
                "raster=%d xcd=%d k_order=%d k_split=%d)" % (
                    d["block_m"], d["block_n"], d["block_k"], d["wave_m"], d["wave_n"],
                    d["mfma_m"], d["mfma_n"], d["mfma_k"], d["lds_stages"], d["lds_pad"],
                    d["unroll_k"], d["raster"], d["xcd_remap"], d["k_order"], d["k_split"]))


class XtcError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = "%s: %s (status %d)" % (where, xtc_status_str(status), status)
        if status == XTC_ERR_HIP:
            msg += ", hipError %d" % _lib.xtc_last_hip_error()
        super().__init__(msg)


def _load():
    # torch ships its own HIP runtime (same soname as ROCm's).  Loading torch
    # first makes libxtc.so bind to that one runtime; loaded the other way
    # round, the process would map two runtimes, and torch's device memory
    # and streams would be invalid handles for the library's launches.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "libxtc.so is not built (expected at %s); run `python paper_2512_16512_amd/build.py`"
            % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    i64, vp, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_int32
    sp = ctypes.POINTER(Sched)
    lib.xtc_matmul.argtypes = [i64, i64, i64, vp, i64, vp, i64, vp, i64, i32, sp, vp]
    lib.xtc_matmul.restype = i32
    lib.xtc_conv2d_nchw.argtypes = [i64] * 11 + [vp, vp, vp, i32, sp, vp]
    lib.xtc_conv2d_nchw.restype = i32
    lib.xtc_matmul_relu.argtypes = lib.xtc_matmul.argtypes
    lib.xtc_matmul_relu.restype = i32
    lib.xtc_conv2d_nchw_relu.argtypes = lib.xtc_conv2d_nchw.argtypes
    lib.xtc_conv2d_nchw_relu.restype = i32
    lib.xtc_default_schedule.argtypes = [i32, i32, i64, i64, i64, sp]
    lib.xtc_default_schedule.restype = i32
    lib.xtc_sched_check.argtypes = [i32, i32, sp]
    lib.xtc_sched_check.restype = i32
    lib.xtc_sched_occupancy.argtypes = [i32, i32, i64, sp, ctypes.POINTER(i32)]
    lib.xtc_sched_occupancy.restype = i32
    lib.xtc_sched_list.argtypes = [i32, i32, sp, i32]
    lib.xtc_sched_list.restype = i32
    lib.xtc_status_str.argtypes = [i32]
    lib.xtc_status_str.restype = ctypes.c_char_p
    lib.xtc_last_hip_error.argtypes = []
    lib.xtc_last_hip_error.restype = i32
    lib.xtc_conv_max_k.argtypes = []
    lib.xtc_conv_max_k.restype = i64
    lib.xtc_version.argtypes = []
    lib.xtc_version.restype = i32
    return lib


_lib = _load()

# Every symbol include/xtc.h declares.
EXPORTS = ("xtc_matmul", "xtc_conv2d_nchw", "xtc_matmul_relu", "xtc_conv2d_nchw_relu",
           "xtc_default_schedule", "xtc_sched_occupancy", "xtc_sched_check",
           "xtc_sched_list", "xtc_status_str", "xtc_last_hip_error", "xtc_conv_max_k",
           "xtc_version")


def _sp(sched):
    return ctypes.byref(sched) if sched is not None else None


# ------------------------------------------------------------- raw C ABI


def xtc_matmul(M, N, K, A, lda, B, ldb, C, ldc, dtype, sched=None, stream=0) -> int:
    return _lib.xtc_matmul(M, N, K, A, lda, B, ldb, C, ldc, dtype, _sp(sched), stream)


def xtc_conv2d_nchw(N, C, H, W, OC, R, S, stride_h, stride_w, pad_h, pad_w, X, Wt, Y, dtype,
                    sched=None, stream=0) -> int:
    return _lib.xtc_conv2d_nchw(N, C, H, W, OC, R, S, stride_h, stride_w, pad_h, pad_w, X, Wt, Y,
                                dtype, _sp(sched), stream)


def xtc_matmul_relu(M, N, K, A, lda, B, ldb, C, ldc, dtype, sched=None, stream=0) -> int:
    return _lib.xtc_matmul_relu(M, N, K, A, lda, B, ldb, C, ldc, dtype, _sp(sched), stream)


def xtc_conv2d_nchw_relu(N, C, H, W, OC, R, S, stride_h, stride_w, pad_h, pad_w, X, Wt, Y, dtype,
                         sched=None, stream=0) -> int:
    return _lib.xtc_conv2d_nchw_relu(N, C, H, W, OC, R, S, stride_h, stride_w, pad_h, pad_w, X,
                                     Wt, Y, dtype, _sp(sched), stream)


def xtc_default_schedule(op, dtype, M, N, K) -> Sched:
    s = Sched()
    st = _lib.xtc_default_schedule(op, dtype, M, N, K, ctypes.byref(s))
    if st != XTC_OK:
        raise XtcError(st, "xtc_default_schedule")
    return s


def xtc_sched_check(op, dtype, sched) -> int:
    return _lib.xtc_sched_check(op, dtype, _sp(sched))


def xtc_sched_occupancy(op, dtype, K, sched) -> int:
    """Workgroups of the instance ``sched`` names that one CU holds at once."""
    n = ctypes.c_int32(0)
    st = _lib.xtc_sched_occupancy(op, dtype, K, _sp(sched), ctypes.byref(n))
    if st != XTC_OK:
        raise XtcError(st, "xtc_sched_occupancy")
    return n.value


def xtc_sched_list(op, dtype):
    n = _lib.xtc_sched_list(op, dtype, None, 0)
    if n < 0:
        return []
    arr = (Sched * n)()
    _lib.xtc_sched_list(op, dtype, arr, n)
    return list(arr)


def xtc_status_str(status) -> str:
    return _lib.xtc_status_str(status).decode()


def xtc_last_hip_error() -> int:
    return _lib.xtc_last_hip_error()


def xtc_conv_max_k() -> int:
    return _lib.xtc_conv_max_k()


def xtc_version() -> int:
    return _lib.xtc_version()


# ------------------------------------------------------- torch conveniences


def _stream(torch, device):
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(torch, t):
    if t.dtype == torch.float32:
        return XTC_F32
    if t.dtype == torch.bfloat16:
        return XTC_BF16
    raise TypeError("unsupported dtype %s (float32 or bfloat16)" % t.dtype)


def _check_rowmajor(t, name):
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError("%s must be a 2-D row-major tensor (unit column stride)" % name)


def matmul(a, b, out=None, sched=None, relu=False):
    """``out = a @ b`` on the GPU (``relu(a @ b)`` fused when ``relu``).
    ``a`` [M,K] and ``b`` [K,N] are both float32 or both bfloat16 CUDA tensors
    with unit column stride; ``out`` is float32 [M,N] (allocated when None).
    Enqueued on torch's current stream."""
    import torch
    _check_rowmajor(a, "a")
    _check_rowmajor(b, "b")
    if a.dtype != b.dtype:
        raise TypeError("a and b must have the same dtype")
    if not (a.is_cuda and b.is_cuda):
        raise ValueError("a and b must be CUDA (HIP) tensors")
    M, K = a.shape
    K2, N = b.shape
    if K2 != K:
        raise ValueError("inner dimensions differ: %d vs %d" % (K, K2))
    if out is None:
        out = torch.empty((M, N), dtype=torch.float32, device=a.device)
    _check_rowmajor(out, "out")
    if out.dtype != torch.float32 or tuple(out.shape) != (M, N):
        raise ValueError("out must be float32 [M, N]")
    lda = a.stride(0) if M > 1 else max(K, 1)
    ldb = b.stride(0) if K > 1 else max(N, 1)
    ldc = out.stride(0) if M > 1 else max(N, 1)
    fn = xtc_matmul_relu if relu else xtc_matmul
    st = fn(M, N, K, a.data_ptr(), lda, b.data_ptr(), ldb, out.data_ptr(), ldc,
            _dtype_code(torch, a), sched, _stream(torch, a.device))
    if st != XTC_OK:
        raise XtcError(st, fn.__name__)
    return out


def conv2d_nchw(x, w, stride=1, pad=0, out=None, sched=None, relu=False):
    """Zero-padded cross-correlation of NCHW ``x`` with OIHW ``w`` (both
    float32 or both bfloat16, contiguous CUDA tensors) into a float32 NCHW
    ``out`` (relu fused into the epilogue when ``relu``)."""
    import torch
    if x.dim() != 4 or w.dim() != 4 or not x.is_contiguous() or not w.is_contiguous():
        raise ValueError("x and w must be contiguous 4-D tensors")
    if x.dtype != w.dtype:
        raise TypeError("x and w must have the same dtype")
    N, C, H, W = x.shape
    OC, C2, R, S = w.shape
    if C2 != C:
        raise ValueError("channel counts differ")
    sh, sw = (stride, stride) if isinstance(stride, int) else stride
    ph, pw = (pad, pad) if isinstance(pad, int) else pad
    OH = (H + 2 * ph - R) // sh + 1
    OW = (W + 2 * pw - S) // sw + 1
    if out is None:
        out = torch.empty((N, OC, max(OH, 0), max(OW, 0)), dtype=torch.float32, device=x.device)
    if not out.is_contiguous() or tuple(out.shape) != (N, OC, OH, OW):
        raise ValueError("out must be a contiguous [N, OC, OH, OW] tensor")
    fn = xtc_conv2d_nchw_relu if relu else xtc_conv2d_nchw
    st = fn(N, C, H, W, OC, R, S, sh, sw, ph, pw, x.data_ptr(), w.data_ptr(), out.data_ptr(),
            _dtype_code(torch, x), sched, _stream(torch, x.device))
    if st != XTC_OK:
        raise XtcError(st, fn.__name__)
    return out
