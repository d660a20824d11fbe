"""GPU parity of the fused-relu entry points and of the paper's other
workloads, through the C ABI, against the fp64 oracle.

relu is the consumer of the paper's matmul+relu graph (Sec. 5.2, Fig. 9); the
oracle applies it to its finished fp64 result.  With small-integer inputs the
products are exact, so every compiled instance must match bit for bit, ragged
edges included; the workloads of Sec. 3.1, 5.2, 6.1 and 6.2 are checked over
every output within the relative Frobenius tolerance.
"""
import numpy as np
import pytest

import oracle
import xtc_inputs as xi
from _helpers import assert_parity, say, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def x():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2512_16512_amd as mod  # raises ImportError if libxtc.so is missing
    return mod


def _prep(A, B, dtype):
    if dtype == "bf16":
        return xi.f32_to_bf16_bits(A), xi.f32_to_bf16_bits(B)
    return A, B


def _mm(x, A, B, relu, sched=None):
    import torch
    c = torch.full((A.shape[0], B.shape[1]), float("nan"), dtype=torch.float32, device="cuda")
    x.matmul(to_dev(A), to_dev(B), out=c, sched=sched, relu=relu)
    return to_host(c)


# --------------------------------------------------------- fused relu, exact


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,N,K", [(300, 264, 200), (65, 33, 1000), (520, 136, 1032)])
def test_matmul_relu_exact_every_instance(x, dtype, M, N, K):
    A, B = _prep(xi.small_int_f32(21, (M, K)), xi.small_int_f32(22, (K, N)), dtype)
    plain = oracle.matmul(A, B)
    ref = oracle.relu(plain)
    assert (plain < 0).mean() > 0.3          # both branches are exercised
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    for s in x.xtc_sched_list(x.XTC_OP_MATMUL, code):
        for raster in (0, 8):
            s.raster = raster
            say("relu", dtype, (M, N, K), s)
            got = _mm(x, A, B, True, sched=s)
            assert np.array_equal(got, ref), "%s %s: relu not bit-exact" % (dtype, s)


@pytest.mark.parametrize("shape", [
    (2, 8, 17, 19, 70, 3, 3, 1, 1),     # channel-major kernels (C % 32 != 0), ragged edges
    (2, 64, 9, 10, 40, 3, 3, 1, 1),     # tap-major kernels
    (1, 3, 30, 30, 16, 7, 7, 2, 3),     # the 7x7 stride-2 shape, scaled down
    (1, 3, 30, 28, 16, 7, 7, 2, 3),     # the same with 16-byte patch rows (width a multiple of 4)
    (1, 16, 56, 56, 40, 3, 3, 1, 1),    # halo-tiled kernel
    (2, 64, 9, 8, 40, 3, 3, 1, 1),      # bf16 row-streaming kernel (C = 64, OW % 4 == 0)
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_conv_relu_exact_every_instance(x, shape, dtype):
    N, C, H, W_, OC, R, S, stride, pad = shape
    X = xi.small_int_f32(23, (N, C, H, W_))
    W = xi.small_int_f32(24, (OC, C, R, S))
    X, W = _prep(X, W, dtype)
    ref = oracle.relu(oracle.conv2d(X, W, stride=stride, pad=pad))
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    for s in x.xtc_sched_list(x.XTC_OP_CONV2D, code):
        say("conv relu", dtype, shape, s)
        got = to_host(x.conv2d_nchw(to_dev(X), to_dev(W), stride=stride, pad=pad, sched=s,
                                    relu=True))
        assert np.array_equal(got, ref), "conv relu %s %s: not bit-exact" % (shape, s)


def test_matmul_relu_hand_worked(x):
    import json
    import os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "matmul_relu_2x3.json")))
    A = np.array(g["A"], np.float32)
    B = np.array(g["B"], np.float32)
    for dtype in ("f32", "bf16"):
        a, b = _prep(A, B, dtype)
        assert np.array_equal(_mm(x, a, b, True), np.array(g["relu_C"], np.float32))
        assert np.array_equal(_mm(x, a, b, False), np.array(g["C"], np.float32))


def test_matmul_relu_ieee_specials(x):
    # inf * 0 gives NaN, which relu keeps; +inf stays, -inf becomes 0.
    M, N, K = 70, 90, 40
    A = xi.small_int_f32(25, (M, K))
    B = xi.small_int_f32(26, (K, N))
    A[3, :] = 0.0
    A[3, 5] = np.inf
    B[5, :] = 0.0
    B[5, 10] = 1.0
    B[5, 11] = -1.0
    ref = oracle.relu(oracle.matmul(A, B))
    assert np.isnan(ref[3, 0]) and ref[3, 10] == np.inf and ref[3, 11] == 0.0
    for s in x.xtc_sched_list(x.XTC_OP_MATMUL, x.XTC_F32):
        say("relu specials", s)
        got = _mm(x, A, B, True, sched=s)
        assert np.array_equal(got, ref, equal_nan=True), "%s" % s


def test_matmul_relu_leading_dims_and_K_zero(x):
    import torch
    M, N, K = 37, 45, 29
    A = xi.small_int_f32(27, (M, K))
    B = xi.small_int_f32(28, (K, N))
    ldc = N + 7
    c = torch.full((M, ldc), 12345.0, dtype=torch.float32, device="cuda")
    a, b = to_dev(A), to_dev(B)
    st = x.xtc_matmul_relu(M, N, K, a.data_ptr(), K, b.data_ptr(), N, c.data_ptr(), ldc,
                           x.XTC_F32)
    assert st == 0
    got = to_host(c)
    assert np.array_equal(got[:, :N], oracle.relu(oracle.matmul(A, B)))
    assert np.all(got[:, N:] == 12345.0)
    st = x.xtc_matmul_relu(M, N, 0, 0, 1, 0, N, c.data_ptr(), ldc, x.XTC_F32)
    assert st == 0
    got = to_host(c)
    assert np.all(got[:, :N] == 0.0) and np.all(got[:, N:] == 12345.0)


def test_relu_and_plain_agree_where_nonnegative(x):
    # the fused path runs the same instance: relu(plain) == fused, bit for bit,
    # on random (not exactly representable) products too
    for dtype in ("f32", "bf16"):
        A, B = _prep(xi.uniform_f32(29, (300, 200)), xi.uniform_f32(30, (200, 264)), dtype)
        plain = _mm(x, A, B, False)
        fused = _mm(x, A, B, True)
        assert np.array_equal(fused, np.where(plain < 0, np.float32(0), plain))


# -------------------------------------------------- the paper's workloads


def _workload_ids():
    return [c["index"] for c in xi.PAPER_WORKLOADS]


@pytest.mark.parametrize("wi", _workload_ids())
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_paper_workload_parity(x, wi, dtype):
    cfg = next(c for c in xi.PAPER_WORKLOADS if c["index"] == wi)
    if cfg["op"] == "conv2d":
        X, W = xi.conv_inputs(cfg)
        if dtype == "bf16":
            X, W = xi.f32_to_bf16_bits(X), xi.f32_to_bf16_bits(W)
        say("workload", cfg["name"], dtype)
        y = x.conv2d_nchw(to_dev(X), to_dev(W), stride=cfg["stride"], pad=cfg["pad"])
        ref = oracle.conv2d(X, W, stride=cfg["stride"], pad=cfg["pad"])
        err = assert_parity(to_host(y), ref, dtype, cfg["name"])
        say("  rel_fro = %.3e" % err)
        yr = x.conv2d_nchw(to_dev(X), to_dev(W), stride=cfg["stride"], pad=cfg["pad"], relu=True)
        err = assert_parity(to_host(yr), oracle.relu(ref), dtype, cfg["name"] + " + relu")
        return
    A, B = _prep(*xi.matmul_inputs(cfg), dtype)
    relu = cfg["op"] == "matmul_relu"
    say("workload", cfg["name"], dtype)
    ref = oracle.matmul(A, B)
    if relu:
        ref = oracle.relu(ref)
    got = _mm(x, A, B, relu)
    err = assert_parity(got, ref, dtype, cfg["name"])
    say("  rel_fro = %.3e" % err)


def test_graph_replay_matches_eager(x):
    # The C ABI launched under HIP graph capture (as the benchmark times the
    # small workloads): every replay, with eager work and synchronisations in
    # between, reproduces the eager result bit for bit.
    import torch
    A = xi.uniform_f32(31, (512, 128))
    B = xi.uniform_f32(32, (128, 1024))
    a, b = to_dev(A), to_dev(B)
    c = torch.empty((512, 1024), dtype=torch.float32, device="cuda")
    eager = x.matmul(a, b, relu=True).clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        x.matmul(a, b, out=c, relu=True)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        for _ in range(3):
            x.matmul(a, b, out=c, relu=True)
    for rep in range(4):
        c.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        say("graph replay", rep)
        assert torch.equal(c, eager), "replay %d differs from the eager result" % rep
    ref = oracle.relu(oracle.matmul(A, B))
    assert_parity(to_host(c), ref, "f32", "graph replay")


def test_every_instance_fits_on_a_cu(x):
    # the occupancy query: every compiled instance has at least one resident
    # workgroup per CU at the reduction lengths it is used with
    for op, dt in ((x.XTC_OP_MATMUL, x.XTC_F32), (x.XTC_OP_MATMUL, x.XTC_BF16),
                   (x.XTC_OP_CONV2D, x.XTC_F32)):
        for s in x.xtc_sched_list(op, dt):
            for K in (1, 576, 4096):
                n = x.xtc_sched_occupancy(op, dt, K, s)
                assert 1 <= n <= 32, (op, dt, K, s, n)
