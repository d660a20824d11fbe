"""Seeded synthetic inputs shared by the oracle side and the GPU side.

This module holds data generation only: no part of the contraction is computed
here.  Both the fp64 oracle and the HIP path receive exactly the arrays these
functions return, so a disagreement between them can never come from the
inputs.

Generator
---------
splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014), used counter-style: element ``i`` of stream ``seed``
is ``mix(seed + (i + 1) * 0x9E3779B97F4A7C15)`` where ``mix`` is the published
finaliser.  A value in [-1, 1) is ``(z >> 40) * 2**-23 - 1``: 24 random bits on
a 2**-23 grid, exactly representable in fp32.

bf16 values are the round-to-nearest-even of those fp32 values on the bit
pattern (finite inputs only, no NaN case).

Seeds follow ``1000 * index + stream`` (the workload's index) with stream 1 = A (or X), 2 = B
(or W), 3 = sample indices.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

_CHUNK = 1 << 20
_THREADS = min(8, os.cpu_count() or 1)


def _mix_chunk(seed_u, lo, hi):
    """splitmix64 outputs for counters lo+1 .. hi (in place, wrapping)."""
    z = np.arange(lo + 1, hi + 1, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z *= GOLDEN
        z += seed_u
        z ^= z >> np.uint64(30)
        z *= _M1
        z ^= z >> np.uint64(27)
        z *= _M2
        z ^= z >> np.uint64(31)
    return z


def _parallel_fill(n, fn):
    """Run ``fn(lo, hi)`` over [0, n) in chunks on a thread pool (numpy
    releases the GIL inside its ufuncs)."""
    starts = range(0, n, _CHUNK)
    if n <= _CHUNK or _THREADS == 1:
        for lo in starts:
            fn(lo, min(n, lo + _CHUNK))
        return
    with ThreadPoolExecutor(_THREADS) as ex:
        list(ex.map(lambda lo: fn(lo, min(n, lo + _CHUNK)), starts))


def splitmix64(seed: int, n: int, start: int = 0) -> np.ndarray:
    """Return ``n`` consecutive outputs of splitmix64 stream ``seed``.

    Output ``i`` (0-based, counting from ``start``) uses state
    ``seed + (start + i + 1) * GOLDEN`` (mod 2**64).
    """
    out = np.empty(n, dtype=np.uint64)
    seed_u = np.uint64(seed & 0xFFFFFFFFFFFFFFFF)

    def fill(lo, hi):
        out[lo:hi] = _mix_chunk(seed_u, start + lo, start + hi)

    _parallel_fill(n, fill)
    return out


def uniform_f32(seed: int, shape) -> np.ndarray:
    """Uniform values in [-1, 1) on a 2**-23 grid, exact in fp32, filled in
    dense (row-major / NCHW / OIHW) order."""
    n = int(np.prod(shape)) if len(shape) else 1
    out = np.empty(n, dtype=np.float32)
    seed_u = np.uint64(seed & 0xFFFFFFFFFFFFFFFF)

    def fill(lo, hi):
        top = (_mix_chunk(seed_u, lo, hi) >> np.uint64(40)).astype(np.float32)
        top *= np.float32(2.0 ** -23)  # exact: 24-bit integer times a power of two
        top -= np.float32(1.0)          # exact: result lies on the 2**-23 grid
        out[lo:hi] = top

    _parallel_fill(n, fill)
    return out.reshape(shape)


def small_int_f32(seed: int, shape, lo: int = -2, hi: int = 2) -> np.ndarray:
    """Integers in [lo, hi] as fp32.  With |entries| <= 2 every partial sum of a
    dot product of length K is an integer of magnitude <= 4K, exact in fp32 for
    K < 2**22, so the result does not depend on summation order."""
    n = int(np.prod(shape)) if len(shape) else 1
    z = splitmix64(seed, n)
    span = np.uint64(hi - lo + 1)
    v = (z % span).astype(np.int64) + lo
    return v.astype(np.float32).reshape(shape)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even of fp32 values to bf16, returned as uint16 bits.
    Inputs must be finite (then ``b + 0x7FFF + lsb`` cannot overflow 32 bits)."""
    src = np.ascontiguousarray(x, dtype=np.float32).reshape(-1).view(np.uint32)
    out = np.empty(src.shape[0], dtype=np.uint16)

    def fill(lo, hi):
        b = src[lo:hi].copy()
        lsb = (b >> np.uint32(16)) & np.uint32(1)
        b += np.uint32(0x7FFF)
        b += lsb
        b >>= np.uint32(16)
        out[lo:hi] = b

    _parallel_fill(src.shape[0], fill)
    return out.reshape(np.shape(x))


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).reshape(np.shape(bits))


def sample_indices_matmul(seed: int, M: int, N: int, count: int = 4096):
    """``count`` (i, j) output positions drawn with replacement:
    ``i = (z >> 32) % M``, ``j = (z & 0xFFFFFFFF) % N``."""
    z = splitmix64(seed, count)
    i = ((z >> np.uint64(32)) % np.uint64(M)).astype(np.int64)
    j = ((z & np.uint64(0xFFFFFFFF)) % np.uint64(N)).astype(np.int64)
    return i, j


def sample_indices_flat(seed: int, total: int, count: int = 4096) -> np.ndarray:
    """``count`` flat output indices ``z % total`` drawn with replacement."""
    z = splitmix64(seed, count)
    return (z % np.uint64(total)).astype(np.int64)


def seed(index: int, stream: int) -> int:
    """Seed of stream `stream` of workload `index`: 1 = A/X, 2 = B/W,
    3 = sample indices."""
    return 1000 * index + stream


# The five synthetic workloads.  "check" is "full" when every output is
# compared, else the number of seeded sampled outputs; "index" numbers the
# workload for its seeds.
WORKLOADS = [
    dict(index=0, op="matmul", dtype="f32", M=256, N=256, K=256, check="full",
         name="matmul fp32 256x256x256"),
    dict(index=1, op="matmul", dtype="f32", M=1000, N=1000, K=1000, check="full",
         name="matmul fp32 1000x1000x1000 (ragged)"),
    dict(index=2, op="matmul", dtype="f32", M=4096, N=4096, K=4096, check=4096,
         name="matmul fp32 4096x4096x4096"),
    dict(index=3, op="matmul", dtype="bf16", M=8192, N=8192, K=8192, check=4096,
         name="matmul bf16-in fp32-acc 8192x8192x8192"),
    dict(index=4, op="conv2d", dtype="f32", N=32, C=64, H=56, W=56, OC=64, R=3, S=3,
         stride=1, pad=1, check=4096,
         name="conv2d NCHW fp32 32x64x56x56 -> 64, 3x3, stride 1, pad 1"),
]
MATMUL_F32_256, MATMUL_F32_1000, MATMUL_F32_4096, MATMUL_BF16_8192, CONV_F32_56 = WORKLOADS

# A tall-skinny product (16 output columns): 8 FLOP per algorithmic byte, far
# below the fp32 ridge point, so it measures the path's HBM streaming rate.
MATMUL_F32_SKINNY = dict(index=10, op="matmul", dtype="f32", M=32768, N=16, K=4096, check=4096,
                         name="matmul fp32 32768x16x4096 (tall-skinny)")


# The other workloads the paper runs, as extra parity and measurement cases.
# Same generators; seeds follow the index.  "matmul_relu" is the matmul with
# its consumer relu fused (the graph of the paper's strategy example).
PAPER_WORKLOADS = [
    dict(index=5, op="matmul", dtype="f32", M=1024, N=1024, K=1024, check="full",
         name="matmul fp32 1024x1024x1024 (Sec. 6.1)"),
    dict(index=6, op="matmul", dtype="f32", M=512, N=1024, K=128, check="full",
         name="matmul fp32 [512,128]x[128,1024] (Sec. 6.2)"),
    dict(index=7, op="matmul_relu", dtype="f32", M=256, N=1024, K=128, check="full",
         name="matmul+relu fp32 [256,128]x[128,1024] (Sec. 5.2)"),
    dict(index=8, op="matmul", dtype="f32", M=256, N=258, K=512, check="full",
         name="matmul fp32 256x258x512 (Sec. 3.1 running example)"),
    dict(index=9, op="conv2d", dtype="f32", N=1, C=3, H=224, W=224, OC=16, R=7, S=7,
         stride=2, pad=3, check="full",
         name="conv2d NCHW fp32 1x3x224x224 -> 16, 7x7, stride 2, pad 3 (Sec. 6.2)"),
]


def matmul_inputs(cfg: dict):
    """A[M,K], B[K,N] for a matmul config: fp32 arrays, or bf16 bit arrays
    (uint16) when ``cfg['dtype'] == 'bf16'``."""
    c = cfg["index"]
    A = uniform_f32(seed(c, 1), (cfg["M"], cfg["K"]))
    B = uniform_f32(seed(c, 2), (cfg["K"], cfg["N"]))
    if cfg["dtype"] == "bf16":
        return f32_to_bf16_bits(A), f32_to_bf16_bits(B)
    return A, B


def conv_out_hw(H, W, R, S, stride_h, stride_w, pad_h, pad_w):
    """Output spatial size of a zero-padded, undilated conv2d."""
    return ((H + 2 * pad_h - R) // stride_h + 1, (W + 2 * pad_w - S) // stride_w + 1)


def conv_inputs(cfg: dict):
    """X[N,C,H,W] and W[OC,C,R,S] for a conv config (fp32)."""
    c = cfg["index"]
    X = uniform_f32(seed(c, 1), (cfg["N"], cfg["C"], cfg["H"], cfg["W"]))
    Wt = uniform_f32(seed(c, 2), (cfg["OC"], cfg["C"], cfg["R"], cfg["S"]))
    return X, Wt
