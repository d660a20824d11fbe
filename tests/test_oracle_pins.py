"""Pins of the fp64 oracle against facts fixed by the paper and by mathematics.

Matmul follows the paper's untransformed loop nest (Sec. 3.1, Fig. 2); conv2d is
read as zero-padded cross-correlation (NCHW, OIHW).  Every pin here is
independent of the oracle's own code: hand-worked values, closed forms, exact
integer arithmetic, or a library routine in float64.
"""
import ctypes
import json
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import xtc_inputs as xi

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    return json.load(open(os.path.join(GOLDEN, name)))


# ------------------------------------------------------------------ matmul


@pytest.mark.parametrize("name", ["matmul_2x2.json", "matmul_3x3.json"])
def test_matmul_hand_worked(name):
    g = _golden(name)
    A = np.array(g["A"], np.float32)
    B = np.array(g["B"], np.float32)
    assert np.array_equal(oracle.matmul(A, B), np.array(g["C"], np.float64))


@pytest.mark.parametrize("M,N,K", [(1, 1, 1), (5, 7, 3), (64, 33, 17), (256, 258, 512)])
def test_matmul_identity(M, N, K):
    B = xi.uniform_f32(11, (K, N))
    A = xi.uniform_f32(12, (M, K))
    I_k = np.eye(K, dtype=np.float32)
    # A = I: C == B exactly (fp32 values are exact in fp64 and only one term is non-zero)
    assert np.array_equal(oracle.matmul(I_k[: min(K, K)], B), B.astype(np.float64))
    # B = I: C == A exactly
    assert np.array_equal(oracle.matmul(A, I_k), A.astype(np.float64))


@pytest.mark.parametrize("M,N,K", [(3, 4, 1), (17, 9, 1000), (8, 8, 4096)])
def test_matmul_all_ones(M, N, K):
    C = oracle.matmul(np.ones((M, K), np.float32), np.ones((K, N), np.float32))
    assert np.all(C == float(K))


def test_matmul_rank_one_closed_form():
    rng = np.random.default_rng(0)
    for K in (1, 7, 300):
        u = rng.integers(-3, 4, size=23).astype(np.float32)
        w = rng.integers(-3, 4, size=31).astype(np.float32)
        A = np.repeat(u[:, None], K, axis=1)      # A[i,k] = u_i
        B = np.repeat(w[None, :], K, axis=0)      # B[k,j] = w_j
        C = oracle.matmul(A, B)
        assert np.array_equal(C, K * np.outer(u, w).astype(np.float64))


@pytest.mark.parametrize("M,N,K", [(31, 33, 65), (128, 96, 257), (7, 300, 1000)])
def test_matmul_small_integers_exact(M, N, K):
    A = xi.small_int_f32(21, (M, K))
    B = xi.small_int_f32(22, (K, N))
    ref = A.astype(np.int64) @ B.astype(np.int64)  # exact integer arithmetic
    assert np.array_equal(oracle.matmul(A, B), ref.astype(np.float64))


def test_matmul_vs_numpy_float64():
    for (M, N, K) in [(10, 20, 30), (65, 129, 255), (256, 258, 512)]:
        A = xi.uniform_f32(31, (M, K))
        B = xi.uniform_f32(32, (K, N))
        ref = A.astype(np.float64) @ B.astype(np.float64)
        got = oracle.matmul(A, B)
        # Only summation order differs: |err| <= ~K * 2**-53 * sum|a||b| <= K^2 2**-53
        assert np.max(np.abs(got - ref)) <= K * K * 2.0 ** -52


def test_matmul_within_fp64_bound_of_exact_result():
    # Inputs lie on the 2**-23 grid, so A*2**23 and B*2**23 are integers and the
    # exact product is an integer over 2**46.  The oracle's fp64 sum must be
    # within the standard dot-product bound gamma_K * sum |a_k b_k| of it.
    M, N, K = 6, 5, 777
    A = xi.uniform_f32(41, (M, K))
    B = xi.uniform_f32(42, (K, N))
    Ai = (A.astype(np.float64) * 2.0 ** 23).astype(np.int64)
    Bi = (B.astype(np.float64) * 2.0 ** 23).astype(np.int64)
    got = oracle.matmul(A, B)
    u = 2.0 ** -53
    gamma = K * u / (1 - K * u)
    for i in range(M):
        for j in range(N):
            exact = Fraction(int(sum(int(a) * int(b) for a, b in zip(Ai[i], Bi[:, j]))), 2 ** 46)
            absum = float(np.sum(np.abs(A[i].astype(np.float64) * B[:, j].astype(np.float64))))
            assert abs(Fraction(got[i, j]) - exact) <= Fraction(gamma * absum)


def test_matmul_bf16_bits_equal_widened_fp32():
    A = xi.f32_to_bf16_bits(xi.uniform_f32(51, (40, 70)))
    B = xi.f32_to_bf16_bits(xi.uniform_f32(52, (70, 30)))
    got = oracle.matmul(A, B)
    ref = oracle.matmul(xi.bf16_bits_to_f32(A), xi.bf16_bits_to_f32(B))
    assert np.array_equal(got, ref)
    # and against numpy float64 on the widened values
    ref2 = xi.bf16_bits_to_f32(A).astype(np.float64) @ xi.bf16_bits_to_f32(B).astype(np.float64)
    assert np.max(np.abs(got - ref2)) < 1e-12


def test_matmul_bf16_identity():
    one = np.uint16(0x3F80)
    K = 24
    I_bits = np.where(np.eye(K, dtype=bool), one, np.uint16(0)).astype(np.uint16)
    B = xi.f32_to_bf16_bits(xi.uniform_f32(53, (K, 10)))
    assert np.array_equal(oracle.matmul(I_bits, B), xi.bf16_bits_to_f32(B).astype(np.float64))


def test_matmul_sampled_equals_full_bitwise():
    M, N, K = 129, 257, 300
    A = xi.uniform_f32(61, (M, K))
    B = xi.uniform_f32(62, (K, N))
    full = oracle.matmul(A, B)
    i, j = xi.sample_indices_matmul(63, M, N, 2000)
    assert np.array_equal(oracle.matmul_sampled(A, B, i, j), full[i, j])


def test_matmul_row_slab_equals_full():
    A = xi.uniform_f32(71, (50, 40))
    B = xi.uniform_f32(72, (40, 30))
    full = oracle.matmul(A, B)
    assert np.array_equal(oracle.matmul(A, B, rows=(13, 29)), full[13:29])


def test_matmul_leading_dims_read_and_write_only_the_logical_matrix():
    # Call the C entry point directly with lda > K, ldb > N, ldc > N.  The pad
    # columns of A and B hold NaN (any read of them would poison the result)
    # and the pad columns of C hold a sentinel that must survive.
    lib = oracle._load()
    M, N, K = 9, 11, 13
    lda, ldb, ldc = K + 3, N + 5, N + 2
    A = xi.small_int_f32(81, (M, K))
    B = xi.small_int_f32(82, (K, N))
    Ap = np.full((M, lda), np.nan, np.float32); Ap[:, :K] = A
    Bp = np.full((K, ldb), np.nan, np.float32); Bp[:, :N] = B
    Cp = np.full((M, ldc), -7.0, np.float64)
    rc = lib.xo_matmul_rows(M, N, K, Ap.ctypes.data_as(ctypes.c_void_p), lda,
                            Bp.ctypes.data_as(ctypes.c_void_p), ldb,
                            Cp.ctypes.data_as(ctypes.c_void_p), ldc, 0, 0, M, 0)
    assert rc == 0
    assert np.array_equal(Cp[:, :N], (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64))
    assert np.all(Cp[:, N:] == -7.0)


def test_matmul_K_zero_gives_zeros():
    C = oracle.matmul(np.zeros((4, 0), np.float32), np.zeros((0, 5), np.float32))
    assert C.shape == (4, 5) and np.all(C == 0.0)


# ------------------------------------------------------------------ conv2d


@pytest.mark.parametrize("name", ["conv_3x3_ones.json", "conv_orientation.json", "conv_stride2.json"])
def test_conv_hand_worked(name):
    g = _golden(name)
    X = np.array(g["X"], np.float32)
    W = np.array(g["W"], np.float32)
    Y = oracle.conv2d(X, W, stride=g["stride"], pad=g["pad"])
    assert np.array_equal(Y, np.array(g["Y"], np.float64))


@pytest.mark.parametrize("N,C,H,W,OC,R,S,stride,pad", [
    (2, 3, 7, 9, 4, 3, 3, 1, 1),
    (1, 5, 8, 8, 3, 3, 3, 2, 1),
    (2, 2, 11, 10, 5, 5, 3, 1, 2),
    (1, 3, 16, 16, 4, 7, 7, 2, 3),   # the paper's 7x7 stride-2 shape, scaled down
    (3, 4, 5, 6, 2, 1, 1, 1, 0),
    # separate vertical/horizontal strides and pads, R != S: a swap of
    # (stride_h, stride_w), (pad_h, pad_w) or (R, S) changes every output
    (1, 3, 9, 11, 4, 3, 5, (1, 2), (2, 1)),
    (2, 2, 10, 7, 3, 5, 3, (2, 1), (0, 2)),
    (1, 4, 8, 12, 2, 1, 3, (3, 1), (1, 0)),
])
def test_conv_vs_torch_float64(N, C, H, W, OC, R, S, stride, pad):
    X = xi.uniform_f32(91, (N, C, H, W))
    Wt = xi.uniform_f32(92, (OC, C, R, S))
    ref = torch.nn.functional.conv2d(torch.from_numpy(X).double(), torch.from_numpy(Wt).double(),
                                     stride=stride, padding=pad).numpy()
    got = oracle.conv2d(X, Wt, stride=stride, pad=pad)
    assert got.shape == ref.shape
    assert np.max(np.abs(got - ref)) < 1e-12


def test_conv_all_ones_border_counts():
    C = 64
    X = np.ones((1, C, 6, 7), np.float32)
    Wt = np.ones((2, C, 3, 3), np.float32)
    Y = oracle.conv2d(X, Wt, stride=1, pad=1)
    assert Y[0, 0, 0, 0] == 4 * C and Y[0, 1, 5, 6] == 4 * C      # corners
    assert Y[0, 0, 0, 3] == 6 * C and Y[0, 0, 2, 0] == 6 * C      # edges
    assert np.all(Y[:, :, 1:-1, 1:-1] == 9 * C)                   # interior


def test_conv_delta_reproduces_input():
    C = 5
    X = xi.uniform_f32(101, (2, C, 9, 8))
    Wt = np.zeros((C, C, 3, 3), np.float32)
    for c in range(C):
        Wt[c, c, 1, 1] = 1.0
    assert np.array_equal(oracle.conv2d(X, Wt, stride=1, pad=1), X.astype(np.float64))


def test_conv_1x1_reduces_to_matmul():
    N, C, H, W, OC = 3, 6, 5, 7, 4
    X = xi.uniform_f32(111, (N, C, H, W))
    Wt = xi.uniform_f32(112, (OC, C, 1, 1))
    Y = oracle.conv2d(X, Wt, stride=1, pad=0)
    for n in range(N):
        ref = oracle.matmul(Wt.reshape(OC, C), X[n].reshape(C, H * W))
        assert np.array_equal(Y[n].reshape(OC, H * W), ref)


def test_conv_sampled_equals_full_bitwise():
    X = xi.uniform_f32(121, (2, 3, 10, 12))
    Wt = xi.uniform_f32(122, (4, 3, 3, 3))
    full = oracle.conv2d(X, Wt, stride=1, pad=1)
    F = xi.sample_indices_flat(123, full.size, 500)
    assert np.array_equal(oracle.conv2d_sampled(X, Wt, F, stride=1, pad=1), full.ravel()[F])


def test_conv_bf16_equals_widened():
    X = xi.f32_to_bf16_bits(xi.uniform_f32(131, (1, 3, 6, 6)))
    Wt = xi.f32_to_bf16_bits(xi.uniform_f32(132, (2, 3, 3, 3)))
    got = oracle.conv2d(X, Wt, stride=1, pad=1)
    ref = oracle.conv2d(xi.bf16_bits_to_f32(X), xi.bf16_bits_to_f32(Wt), stride=1, pad=1)
    assert np.array_equal(got, ref)


def test_rel_fro():
    assert oracle.rel_fro([0.0, 0.0], [0.0, 0.0]) == 0.0
    assert oracle.rel_fro([1.0], [0.0]) == float("inf")
    assert abs(oracle.rel_fro([3.0, 4.0 + 1e-3], [3.0, 4.0]) - 1e-3 / 5.0) < 1e-15


# -------------------------------------------------------------------- relu
# The consumer of the paper's matmul+relu graph (Sec. 5.2, Fig. 9), fused into
# the contraction's epilogue on the GPU; the oracle applies it to the finished
# fp64 result.


def relu_battery(relu_fn):
    """Pins of relu(v) = (v < 0 ? 0 : v); raises AssertionError on a mismatch.
    Shared with the planted-mistake test, which must see it fail."""
    g = _golden("matmul_relu_2x3.json")
    A = np.array(g["A"], np.float32)
    B = np.array(g["B"], np.float32)
    C = oracle.matmul(A, B)
    assert np.array_equal(C, np.array(g["C"], np.float64))
    assert np.array_equal(relu_fn(C), np.array(g["relu_C"], np.float64))
    # against the library routine in float64, specials included
    v = np.concatenate([xi.uniform_f32(141, (1000,)).astype(np.float64) * 1e3,
                        [0.0, -0.0, np.inf, -np.inf, np.nan, 1e-300, -1e-300]])
    ref = torch.nn.functional.relu(torch.from_numpy(v)).numpy()
    assert np.array_equal(relu_fn(v), ref, equal_nan=True)
    # closed forms: relu(v) - relu(-v) == v and relu(v) + relu(-v) == |v|
    w = xi.uniform_f32(142, (777,)).astype(np.float64)
    assert np.array_equal(relu_fn(w) - relu_fn(-w), w)
    assert np.array_equal(relu_fn(w) + relu_fn(-w), np.abs(w))


def test_relu_pins():
    relu_battery(oracle.relu)


def test_conv_relu_vs_torch_float64():
    X = xi.uniform_f32(143, (2, 3, 9, 9))
    Wt = xi.uniform_f32(144, (4, 3, 3, 3))
    ref = torch.relu(torch.nn.functional.conv2d(torch.from_numpy(X).double(),
                                                torch.from_numpy(Wt).double(), stride=2,
                                                padding=1)).numpy()
    got = oracle.relu(oracle.conv2d(X, Wt, stride=2, pad=1))
    assert np.max(np.abs(got - ref)) < 1e-12
    assert (got == 0).mean() > 0.2      # the case really exercises the negative branch
