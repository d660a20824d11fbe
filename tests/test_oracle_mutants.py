"""Planted mistakes: each edited copy of the oracle source must fail a pin.

The edits are made on the CPU, in a temporary copy of ``oracle/oracle.c``; the
real oracle is never modified.  Each mutant models a plausible slip (a dropped
term, a wrong sign or index, a transposed operand, a wrong padding offset, a
wrong bf16 widening) and must be caught by the battery below, which uses only
hand-worked values, closed forms and exact integer arithmetic.
"""
import ctypes
import json
import os
import shutil
import tempfile

import numpy as np
import pytest

import oracle
from oracle import build as obuild
import xtc_inputs as xi

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

MUTANTS = {
    "transposed_B": ("acc[j] += a * load_elem(B, k * ldb + j, is_bf16);",
                     "acc[j] += a * load_elem(B, j * ldb + k, is_bf16);"),
    "dropped_last_k": ("for (int64_t k = 0; k < K; ++k) {\n                double a",
                       "for (int64_t k = 0; k + 1 < K; ++k) {\n                double a"),
    "wrong_sign": ("acc[j] += a * load_elem", "acc[j] -= a * load_elem"),
    "accumulate_not_overwrite": ("for (int64_t j = 0; j < N; ++j) acc[j] = 0.0;",
                                 "for (int64_t j = 0; j < N; ++j) acc[j] = C[i * ldc + j];"),
    "sampled_swapped_ij": ("load_elem(A, I[s] * lda + k, is_bf16) *",
                           "load_elem(A, J[s] * lda + k, is_bf16) *"),
    "conv_flipped_kernel": ("((oc * C + ic) * R + kh) * S + kw",
                            "((oc * C + ic) * R + (R - 1 - kh)) * S + (S - 1 - kw)"),
    "conv_pad_sign": ("int64_t ih = oh * sh - ph + kh;", "int64_t ih = oh * sh + ph + kh;"),
    "conv_dropped_channel": ("for (int64_t ic = 0; ic < C; ++ic)\n        for (int64_t kh",
                             "for (int64_t ic = 1; ic < C; ++ic)\n        for (int64_t kh"),
    "conv_transposed_hw": ("((n * C + ic) * H + ih) * W + iw", "((n * C + ic) * H + iw) * W + ih"),
    "bf16_wrong_widening": ("((uint32_t)bits) << 16", "((uint32_t)bits) << 15"),
}


def _g(name):
    return json.load(open(os.path.join(GOLDEN, name)))


def _battery(lib):
    """Return the names of the pins that fail for ``lib``."""
    failed = []

    def check(name, ok):
        if not ok:
            failed.append(name)

    for fx in ("matmul_2x2.json", "matmul_3x3.json"):
        g = _g(fx)
        C = oracle.matmul(np.array(g["A"], np.float32), np.array(g["B"], np.float32), lib=lib)
        check(fx, np.array_equal(C, np.array(g["C"], np.float64)))
    K = 9
    B = xi.small_int_f32(1, (K, 7))
    check("identity", np.array_equal(oracle.matmul(np.eye(K, dtype=np.float32), B, lib=lib),
                                     B.astype(np.float64)))
    check("ones", np.all(oracle.matmul(np.ones((3, 40), np.float32), np.ones((40, 5), np.float32),
                                       lib=lib) == 40.0))
    A = xi.small_int_f32(2, (11, 13))
    B = xi.small_int_f32(3, (13, 12))
    full = oracle.matmul(A, B, lib=lib)
    exact = (A.astype(np.int64) @ B.astype(np.int64)).astype(np.float64)
    check("small_int", np.array_equal(full, exact))
    i, j = xi.sample_indices_matmul(4, 11, 12, 64)
    check("sampled", np.array_equal(oracle.matmul_sampled(A, B, i, j, lib=lib), exact[i, j]))
    # overwrite semantics: results written into a buffer that already holds
    # values must not depend on those values
    Cpre = np.full((11, 12), 5.0, np.float64)
    rc = lib.xo_matmul_rows(11, 12, 13, A.ctypes.data_as(ctypes.c_void_p), 13,
                            B.ctypes.data_as(ctypes.c_void_p), 12,
                            Cpre.ctypes.data_as(ctypes.c_void_p), 12, 0, 0, 11, 0)
    check("overwrite", rc == 0 and np.array_equal(Cpre, exact))
    bitsA = xi.f32_to_bf16_bits(np.array([[1.5, -2.0]], np.float32))
    bitsB = xi.f32_to_bf16_bits(np.array([[2.0], [0.25]], np.float32))
    check("bf16", np.array_equal(oracle.matmul(bitsA, bitsB, lib=lib), np.array([[2.5]])))
    for fx in ("conv_3x3_ones.json", "conv_orientation.json", "conv_stride2.json"):
        g = _g(fx)
        Y = oracle.conv2d(np.array(g["X"], np.float32), np.array(g["W"], np.float32),
                          stride=g["stride"], pad=g["pad"], lib=lib)
        check(fx, np.array_equal(Y, np.array(g["Y"], np.float64)))
    X = np.ones((1, 4, 5, 6), np.float32)
    W = np.ones((1, 4, 3, 3), np.float32)
    Y = oracle.conv2d(X, W, stride=1, pad=1, lib=lib)
    check("conv_ones_corner", Y[0, 0, 0, 0] == 16 and Y[0, 0, 2, 2] == 36)
    Xa = xi.small_int_f32(5, (1, 2, 4, 7))
    Wd = np.zeros((2, 2, 3, 3), np.float32)
    Wd[0, 0, 1, 1] = Wd[1, 1, 1, 1] = 1.0
    check("conv_delta", np.array_equal(oracle.conv2d(Xa, Wd, stride=1, pad=1, lib=lib),
                                       Xa.astype(np.float64)))
    return failed


def test_real_oracle_passes_battery():
    assert _battery(oracle._load()) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name):
    if shutil.which(os.environ.get("CC", "gcc")) is None:
        pytest.skip("no host C compiler")
    src = open(obuild.SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) >= 1, "mutation site vanished: %s" % name
    mutated = src.replace(old, new, 1)
    with tempfile.TemporaryDirectory() as d:
        csrc = os.path.join(d, "oracle_mut.c")
        open(csrc, "w").write(mutated)
        lib_path = obuild.build(src=csrc, out=os.path.join(d, "liboracle_mut.so"))
        lib = oracle._load(lib_path)
        failed = _battery(lib)
    assert failed, "planted mistake %r was not caught by any pin" % name


RELU_MUTANTS = {
    "relu_abs": np.abs,
    "relu_min": lambda v: np.minimum(np.asarray(v, np.float64), 0.0),
    "relu_identity": lambda v: np.asarray(v, np.float64),
    "relu_nan_to_zero": lambda v: np.where(np.asarray(v, np.float64) > 0.0, v, 0.0),
    "relu_shifted": lambda v: np.where(np.asarray(v, np.float64) < 1e-7, 0.0, v),
}


@pytest.mark.parametrize("name", sorted(RELU_MUTANTS))
def test_relu_mutant_is_caught(name):
    from tests.test_oracle_pins import relu_battery
    with pytest.raises(AssertionError):
        relu_battery(RELU_MUTANTS[name])
