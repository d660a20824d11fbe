"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Exact cases (small-integer inputs, identity, all-ones, rank-1, conv delta)
must match bit for bit; random uniform inputs must be within the relative
Frobenius tolerance (1e-5 fp32, 1e-2 bf16 inputs) over every output, or over
4096 seeded sampled outputs at the full benchmark sizes (the same default
schedule and launch that bench.py times).
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


def _bits(a):
    return xi.f32_to_bf16_bits(a)


def _prep(A, B, dtype):
    """Host operands for the oracle and the device, for dtype f32 / bf16."""
    if dtype == "bf16":
        A, B = _bits(A), _bits(B)
    return A, B


def _run_mm(x, A, B, sched=None):
    import torch
    a, b = to_dev(A), to_dev(B)
    c = torch.full((A.shape[0], B.shape[1]), float("nan"), dtype=torch.float32, device="cuda")
    x.matmul(a, b, out=c, sched=sched)
    return to_host(c)


# ---------------------------------------------------------- full workloads


@pytest.mark.parametrize("ci", [0, 1, 2, 3, 10])
def test_matmul_workload_parity(x, ci):
    import torch
    cfg = xi.MATMUL_F32_SKINNY if ci == 10 else xi.WORKLOADS[ci]
    say("matmul workload", ci, cfg["name"])
    A, B = xi.matmul_inputs(cfg)
    a, b = to_dev(A), to_dev(B)
    c = x.matmul(a, b)
    if cfg["check"] == "full":
        ref = oracle.matmul(A, B)
        got = to_host(c)
    else:
        i, j = xi.sample_indices_matmul(xi.seed(ci, 3), cfg["M"], cfg["N"], cfg["check"])
        ref = oracle.matmul_sampled(A, B, i, j)
        got = to_host(c[torch.from_numpy(i).cuda(), torch.from_numpy(j).cuda()])
    err = assert_parity(got, ref, cfg["dtype"], cfg["name"])
    say("  rel_fro = %.3e" % err)


@pytest.mark.parametrize("shape", [
    (3, 5, 13, 11, 7, 3, 3, 1, 1),      # C*R*S = 45: scalar weight loads
    (2, 8, 17, 19, 70, 3, 3, 1, 1),     # C*R*S = 72, OC = 70: ragged weight rows, pixel tail
    (3, 16, 9, 14, 64, 3, 3, 2, 1),     # stride 2
    (1, 4, 20, 20, 33, 5, 5, 1, 2),     # 5x5, pad 2
    (2, 12, 11, 7, 16, 1, 1, 1, 0),     # 1x1
    (1, 3, 30, 30, 16, 7, 7, 2, 3),     # the 7x7 stride-2 shape, scaled down
    (1, 64, 12, 12, 130, 3, 3, 1, 1),   # OC > 128: several weight tiles
    (1, 16, 56, 56, 64, 3, 3, 1, 1),    # halo-tiled kernel: 56-wide rows, last tile ragged
    (2, 32, 54, 52, 70, 3, 3, 1, 1),    # halo: OC = 70 (ragged second weight tile), two stages
    (1, 16, 57, 56, 20, 3, 3, 1, 0),    # halo: no padding (55 x 54 output)
    (1, 48, 56, 58, 16, 3, 3, 1, 2),    # halo: pad 2 (60-wide output rows), three stages
    (1, 64, 56, 56, 64, 3, 3, 1, 1),    # halo: four stages (both register sets twice)
    (1, 80, 21, 56, 40, 3, 3, 1, 1),    # halo: five stages, OC = 40
    (2, 64, 9, 8, 40, 3, 3, 1, 1),      # rows: 8-pixel rows, OC = 40 (partial channel tile)
    (1, 64, 7, 58, 128, 3, 3, 1, 0),    # rows: no padding, 5 output rows, two channel tiles
    (3, 64, 13, 54, 16, 3, 3, 1, 2),    # rows: pad 2 (56-wide output), OC = 16
    (1, 64, 56, 56, 70, 3, 3, 1, 1),    # rows: OC = 70
    (2, 64, 3, 4, 64, 3, 3, 1, 1),      # rows: 4 x 4 output, band taller than the image
    (16, 64, 40, 16, 64, 3, 3, 1, 1),   # rows: bands of 3 rows (last step half used)
    (32, 64, 30, 8, 64, 3, 3, 1, 1),    # rows: bands of 4 rows, shorter last band
    (100, 64, 60, 8, 64, 3, 3, 1, 1),   # rows: bands of 20 rows (five steps: both register sets twice)
    (64, 64, 26, 8, 40, 3, 3, 1, 1),    # rows: bands of 7 rows (last step has three), OC = 40
    (64, 64, 21, 10, 64, 3, 3, 1, 0),   # rows: no padding, bands of 5 rows (two steps, one row in the last)
])
def test_conv_bf16_small_int_exact_every_instance(x, shape):
    N, C, H, W_, OC, R, S, stride, pad = shape
    X = xi.f32_to_bf16_bits(xi.small_int_f32(11, (N, C, H, W_)))
    W = xi.f32_to_bf16_bits(xi.small_int_f32(12, (OC, C, R, S)))
    ref = oracle.conv2d(X, W, stride=stride, pad=pad)
    for s in x.xtc_sched_list(x.XTC_OP_CONV2D, x.XTC_BF16):
        for raster in (0, 8):
            s.raster = raster
            say("conv bf16 exact", shape, s)
            got = to_host(x.conv2d_nchw(to_dev(X), to_dev(W), stride=stride, pad=pad, sched=s))
            assert np.array_equal(got, ref), "conv bf16 %s %s: not bit-exact" % (shape, s)


def test_conv_bf16_config_shape_parity(x):
    # the 32x64x56x56 -> 64 layer with bf16 inputs, checked on sampled outputs
    import torch
    cfg = xi.CONV_F32_56
    X, W = xi.conv_inputs(cfg)
    Xb, Wb = xi.f32_to_bf16_bits(X), xi.f32_to_bf16_bits(W)
    say("conv bf16 config shape")
    y = x.conv2d_nchw(to_dev(Xb), to_dev(Wb), stride=cfg["stride"], pad=cfg["pad"])
    F = xi.sample_indices_flat(xi.seed(4, 3), y.numel(), cfg["check"])
    ref = oracle.conv2d_sampled(Xb, Wb, F, stride=cfg["stride"], pad=cfg["pad"])
    got = to_host(y.reshape(-1)[torch.from_numpy(F).cuda()])
    err = assert_parity(got, ref, "bf16", "conv bf16 32x64x56x56")
    say("  rel_fro = %.3e" % err)


def test_conv_config_parity(x):
    import torch
    cfg = xi.CONV_F32_56
    say("conv config", cfg["name"])
    X, W = xi.conv_inputs(cfg)
    y = x.conv2d_nchw(to_dev(X), to_dev(W), stride=cfg["stride"], pad=cfg["pad"])
    F = xi.sample_indices_flat(xi.seed(4, 3), y.numel(), cfg["check"])
    ref = oracle.conv2d_sampled(X, W, F, stride=cfg["stride"], pad=cfg["pad"])
    got = to_host(y.reshape(-1)[torch.from_numpy(F).cuda()])
    err = assert_parity(got, ref, "f32", cfg["name"])
    say("  rel_fro = %.3e" % err)


# ------------------------------------------------- exact, every instance


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("M,N,K", [(300, 200, 150), (128, 256, 64), (65, 33, 1000), (300, 264, 200), (520, 136, 1032)])
def test_small_int_exact_every_instance(x, dtype, M, N, K):
    A, B = _prep(xi.small_int_f32(7, (M, K)), xi.small_int_f32(8, (K, N)), dtype)
    ref = oracle.matmul(A, B)
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    for s in x.xtc_sched_list(x.XTC_OP_MATMUL, code):
        for raster, xcd in ((0, 1), (8, 1), (1, 0)):
            s.raster, s.xcd_remap = raster, xcd
            say(dtype, (M, N, K), s)
            got = _run_mm(x, A, B, sched=s)
            assert np.array_equal(got, ref), "%s %s: not bit-exact" % (dtype, s)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_large_tiles_exact_at_scale(x, dtype):
    """Every instance with 128- or 256-wide tiles on 2048 x 2048 x 4096 small
    integers (exact in fp32 for any summation order): many full interior
    tiles, every CU busy, and 64 to 128 turns of the LDS ring, compared with
    the oracle element by element."""
    M, N, K = 2048, 2048, 4096
    A, B = _prep(xi.small_int_f32(31, (M, K)), xi.small_int_f32(32, (K, N)), dtype)
    ref = oracle.matmul(A, B)
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    n = 0
    for s in x.xtc_sched_list(x.XTC_OP_MATMUL, code):
        if s.block_m < 128 or s.block_n < 128:
            continue
        for raster, xcd in ((1, 0), (4, 1)):
            s.raster, s.xcd_remap = raster, xcd
            say(dtype, (M, N, K), s)
            got = _run_mm(x, A, B, sched=s)
            bad = np.argwhere(got != ref)
            assert bad.size == 0, "%s %s: %d outputs differ, first at %s" % (
                dtype, s, len(bad), tuple(bad[0]))
        n += 1
    assert n >= 3


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [
    # N, C, H, W, OC, R, S, (stride_h, stride_w), (pad_h, pad_w)
    (2, 16, 13, 17, 20, 3, 3, (1, 1), (1, 2)),      # pad_h != pad_w
    (2, 8, 15, 16, 24, 3, 3, (1, 2), (1, 1)),       # stride_h != stride_w
    (1, 12, 14, 13, 17, 3, 5, (1, 1), (1, 2)),      # R != S
    (1, 32, 11, 12, 40, 5, 3, (2, 1), (2, 0)),      # R != S, both asymmetric, tap-major fp32
    (1, 16, 20, 57, 64, 3, 3, (1, 1), (1, 3)),      # halo kernels: pad_w 3, W + pad_w = 60
    (1, 16, 19, 56, 64, 3, 3, (1, 1), (2, 4)),      # halo kernels: pad_w 4, W + pad_w = 60
    (1, 32, 18, 56, 64, 3, 3, (1, 1), (0, 2)),      # halo: pad_h 0, pad_w 2
])
def test_conv_asymmetric_exact_every_instance(x, dtype, shape):
    N, C, H, W_, OC, R, S, stride, pad = shape
    X = xi.small_int_f32(41, (N, C, H, W_))
    W = xi.small_int_f32(42, (OC, C, R, S))
    if dtype == "bf16":
        X, W = _bits(X), _bits(W)
    ref = oracle.conv2d(X, W, stride=stride, pad=pad)
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    for s in x.xtc_sched_list(x.XTC_OP_CONV2D, code) + [None]:
        say("conv asym", dtype, shape, s)
        got = to_host(x.conv2d_nchw(to_dev(X), to_dev(W), stride=stride, pad=pad, sched=s))
        assert got.shape == ref.shape
        assert np.array_equal(got, ref), "conv %s %s %s: not bit-exact" % (dtype, shape, s)


@pytest.mark.parametrize("shape", [
    (3, 5, 13, 11, 7, 3, 3, 1, 1),      # C*R*S = 45: not a multiple of 4 (register-staged path)
    (2, 8, 17, 19, 70, 3, 3, 1, 1),     # C*R*S = 72, OC = 70: ragged weight rows, pixel tail
    (3, 16, 9, 14, 64, 3, 3, 2, 1),     # stride 2
    (1, 4, 20, 20, 33, 5, 5, 1, 2),     # 5x5, pad 2, C*R*S = 100
    (2, 12, 11, 7, 16, 1, 1, 1, 0),     # 1x1
    (2, 64, 9, 10, 40, 3, 3, 1, 1),     # C % 32 == 0: tap-major kernel, OC < 64
    (1, 32, 12, 12, 64, 3, 3, 2, 1),    # tap-major, stride 2
    (2, 96, 7, 7, 70, 1, 1, 1, 0),      # tap-major 1x1, three channel chunks, OC > 64
    (1, 16, 56, 56, 64, 3, 3, 1, 1),    # halo-tiled kernel: 56-wide rows, last tile ragged
    (2, 32, 54, 53, 70, 3, 3, 1, 1),    # halo: odd width, OC > 64 with a ragged weight tile
    (1, 16, 57, 55, 20, 3, 3, 1, 0),    # halo: no padding (53 x 55 output)
    (1, 48, 56, 56, 16, 3, 3, 1, 2),    # halo: pad 2 (58-wide output rows), six stages
    (1, 24, 56, 56, 64, 3, 3, 1, 1),    # balanced halo: 8-channel stages, odd stage count
    (1, 8, 61, 59, 64, 3, 3, 1, 1),     # balanced halo: 400-pixel tiles, second half 12 blocks
    (1, 8, 69, 58, 64, 3, 3, 1, 1),     # balanced halo: 401-pixel tiles, second half 13 blocks
    (2, 8, 7, 57, 48, 3, 3, 1, 1),      # balanced halo: 399-pixel tiles, one tile per image
    (1, 3, 30, 28, 16, 7, 7, 2, 3),     # few channels, 16-byte patch rows: 7x7 stride 2, origin 4
    (2, 4, 16, 16, 12, 3, 3, 1, 0),     # 16-byte patch rows, no padding (origin 0), OC = 12
    (1, 2, 12, 16, 16, 3, 3, 1, 4),     # 16-byte patch rows, pad 4 (origin 4, 20-wide output)
])
def test_conv_small_int_exact_every_instance(x, shape):
    N, C, H, W_, OC, R, S, stride, pad = shape
    X = xi.small_int_f32(9, (N, C, H, W_))
    W = xi.small_int_f32(10, (OC, C, R, S))
    ref = oracle.conv2d(X, W, stride=stride, pad=pad)
    for s in x.xtc_sched_list(x.XTC_OP_CONV2D, x.XTC_F32):
        for raster in (0, 1, 8):
            s.raster = raster
            say("conv exact", shape, s)
            got = to_host(x.conv2d_nchw(to_dev(X), to_dev(W), stride=stride, pad=pad, sched=s))
            assert np.array_equal(got, ref), "conv %s %s: not bit-exact" % (shape, s)


# ---------------------------------------------------------- closed forms


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_identity(x, dtype):
    M, K, N = 200, 200, 333
    B = xi.uniform_f32(11, (K, N))
    I = np.eye(K, dtype=np.float32)
    Ih, Bh = _prep(I, B, dtype)
    say("identity", dtype)
    got = _run_mm(x, Ih, Bh)
    Bval = xi.bf16_bits_to_f32(Bh) if dtype == "bf16" else B
    assert np.array_equal(got, Bval)
    A = xi.uniform_f32(12, (M, K))
    Ah, Ih2 = _prep(A, I, dtype)
    got = _run_mm(x, Ah, Ih2)
    Aval = xi.bf16_bits_to_f32(Ah) if dtype == "bf16" else A
    assert np.array_equal(got, Aval)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K", [1, 7, 1000, 4097])
def test_all_ones_gives_K(x, dtype, K):
    A, B = _prep(np.ones((130, K), np.float32), np.ones((K, 70), np.float32), dtype)
    say("ones", dtype, K)
    assert np.all(_run_mm(x, A, B) == float(K))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rank_one(x, dtype):
    rng = np.random.default_rng(3)
    K = 333
    u = rng.integers(-3, 4, size=150).astype(np.float32)
    w = rng.integers(-3, 4, size=170).astype(np.float32)
    A, B = _prep(np.repeat(u[:, None], K, 1), np.repeat(w[None, :], K, 0), dtype)
    say("rank-1", dtype)
    assert np.array_equal(_run_mm(x, A, B), K * np.outer(u, w).astype(np.float64))


@pytest.mark.parametrize("name", ["matmul_2x2.json", "matmul_3x3.json"])
def test_hand_worked(x, name):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", name)))
    A = np.array(g["A"], np.float32)
    B = np.array(g["B"], np.float32)
    for dtype in ("f32", "bf16"):
        Ah, Bh = _prep(A, B, dtype)
        assert np.array_equal(_run_mm(x, Ah, Bh), np.array(g["C"], np.float64))


# -------------------------------------------------------------- edges


def _ragged_cases():
    sizes = [1, 2, 15, 16, 17, 31, 33, 63, 65, 127, 129, 255, 257, 258, 1000]
    rng = np.random.default_rng(2024)
    cases = [(s, s, s) for s in sizes]
    cases += [tuple(int(v) for v in rng.choice(sizes, 3)) for _ in range(30)]
    return cases


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_ragged_sweep_exact(x, dtype):
    for (M, N, K) in _ragged_cases():
        A, B = _prep(xi.small_int_f32(M * 7 + K, (M, K)), xi.small_int_f32(N * 5 + K, (K, N)), dtype)
        say("ragged", dtype, (M, N, K))
        got = _run_mm(x, A, B)
        assert np.array_equal(got, oracle.matmul(A, B)), (dtype, M, N, K)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_paper_running_example_shape(x, dtype):
    # The paper's running example (Fig. 2): I=256, J=258, K=512, row-major;
    # J = 258 leaves a 2-column remainder and makes ldb unaligned to 16 bytes.
    A, B = _prep(xi.uniform_f32(13, (256, 512)), xi.uniform_f32(14, (512, 258)), dtype)
    say("paper shape 256x258x512", dtype)
    got = _run_mm(x, A, B)
    assert_parity(got, oracle.matmul(A, B), dtype, "256x258x512")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("pad", [(5, 3, 7), (8, 8, 8)])
def test_leading_dims_with_guard_bands(x, dtype, pad):
    import torch
    M, N, K = 190, 140, 77
    pa, pb, pc = pad
    A, B = _prep(xi.small_int_f32(15, (M, K)), xi.small_int_f32(16, (K, N)), dtype)
    ref = oracle.matmul(A, B)
    nan_bits = np.uint16(0x7FC0)
    fill = nan_bits if dtype == "bf16" else np.float32(np.nan)
    Ap = np.full((M, K + pa), fill, dtype=A.dtype); Ap[:, :K] = A
    Bp = np.full((K, N + pb), fill, dtype=B.dtype); Bp[:, :N] = B
    ad, bd = to_dev(Ap), to_dev(Bp)
    c = torch.full((M, N + pc), -123.0, dtype=torch.float32, device="cuda")
    say("leading dims", dtype, pad)
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    st = x.xtc_matmul(M, N, K, ad.data_ptr(), K + pa, bd.data_ptr(), N + pb, c.data_ptr(), N + pc,
                      code, None, torch.cuda.current_stream().cuda_stream)
    assert st == 0
    got = to_host(c)
    assert np.array_equal(got[:, :N], ref), "logical C wrong or NaN leaked from the guard bands"
    assert np.all(got[:, N:] == -123.0), "columns N..ldc of C were written"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_K_zero_writes_zeros_and_empty_is_noop(x, dtype):
    import torch
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    a = torch.empty((50, 0), dtype=tdt, device="cuda")
    b = torch.empty((0, 70), dtype=tdt, device="cuda")
    c = torch.full((50, 70), 5.0, device="cuda")
    x.matmul(a, b, out=c)
    assert np.all(to_host(c) == 0.0)
    e = torch.full((0, 70), 5.0, device="cuda")
    x.matmul(torch.empty((0, 3), dtype=tdt, device="cuda"), torch.ones((3, 70), dtype=tdt, device="cuda"), out=e)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_deterministic_and_raster_independent(x, dtype):
    import torch
    A, B = _prep(xi.uniform_f32(17, (1000, 1000)), xi.uniform_f32(18, (1000, 1000)), dtype)
    a, b = to_dev(A), to_dev(B)
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    s = x.xtc_default_schedule(x.XTC_OP_MATMUL, code, 1000, 1000, 1000)
    say("determinism", dtype, s)
    first = to_host(x.matmul(a, b, sched=s))
    for rep in range(20):
        assert np.array_equal(to_host(x.matmul(a, b, sched=s)), first), "run %d differs" % rep
    for raster, xcd in ((0, 0), (1, 1), (3, 1), (16, 0)):
        s.raster, s.xcd_remap = raster, xcd
        assert np.array_equal(to_host(x.matmul(a, b, sched=s)), first), (raster, xcd)
    assert_parity(first, oracle.matmul(A, B), dtype, "1000^3")


# --------------------------------------------------------------- conv


def _conv(x, X, W, stride, pad, sched=None):
    return to_host(x.conv2d_nchw(to_dev(X), to_dev(W), stride=stride, pad=pad, sched=sched))


def test_conv_delta_is_identity(x):
    C = 6
    X = xi.uniform_f32(19, (2, C, 17, 19))
    W = np.zeros((C, C, 3, 3), np.float32)
    for c in range(C):
        W[c, c, 1, 1] = 1.0
    say("conv delta")
    assert np.array_equal(_conv(x, X, W, 1, 1), X.astype(np.float64))


def test_conv_all_ones_borders(x):
    C = 64
    say("conv ones")
    Y = _conv(x, np.ones((2, C, 9, 10), np.float32), np.ones((3, C, 3, 3), np.float32), 1, 1)
    assert np.all(Y[:, :, 0, 0] == 4 * C) and np.all(Y[:, :, -1, -1] == 4 * C)
    assert np.all(Y[:, :, 0, 1:-1] == 6 * C) and np.all(Y[:, :, 1:-1, 0] == 6 * C)
    assert np.all(Y[:, :, 1:-1, 1:-1] == 9 * C)


@pytest.mark.parametrize("name", ["conv_3x3_ones.json", "conv_orientation.json", "conv_stride2.json"])
def test_conv_hand_worked(x, name):
    import json, os
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", name)))
    Y = _conv(x, np.array(g["X"], np.float32), np.array(g["W"], np.float32), g["stride"], g["pad"])
    assert np.array_equal(Y, np.array(g["Y"], np.float64))


@pytest.mark.parametrize("N,C,H,W,OC,R,S,stride,pad", [
    (2, 3, 64, 64, 16, 7, 7, 2, 3),      # the paper's 7x7 stride-2 conv, reduced spatially
    (3, 4, 10, 9, 5, 1, 1, 1, 0),        # 1x1
    (2, 8, 15, 13, 70, 3, 3, 2, 1),      # OC > 64: two tile rows, ragged
    (1, 16, 30, 30, 32, 5, 5, 1, 2),
    (4, 64, 14, 14, 64, 3, 3, 1, 1),
])
def test_conv_shapes_vs_oracle(x, N, C, H, W, OC, R, S, stride, pad):
    X = xi.uniform_f32(20, (N, C, H, W))
    Wt = xi.uniform_f32(21, (OC, C, R, S))
    say("conv", (N, C, H, W, OC, R, S, stride, pad))
    got = _conv(x, X, Wt, stride, pad)
    assert_parity(got, oracle.conv2d(X, Wt, stride=stride, pad=pad), "f32", "conv")
