"""Seeded randomized parity and concurrency checks through the C ABI.

- Random shapes (ragged in every dimension, leading dimensions with padding)
  paired with random compiled instances, raster orders and the relu flag;
  small-integer inputs make every correct result bit-exact.
- Random 3x3 stride-1 layers in and around the class of the patch-staging
  conv kernels, through every such instance and the default schedule.
- A wider seeded sweep over every kind of instance (matmul and conv, both
  dtypes, narrow and long-reduction shapes, misaligned bf16 operands).
- Several host threads, each on its own stream, launching different
  contractions at once: the library keeps no state shared between calls, so
  every result must equal its single-threaded one.
"""
import threading

import numpy as np
import pytest

import oracle
import xtc_inputs as xi
from _helpers import say, to_dev, to_host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def x():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    import paper_2512_16512_amd as mod
    return mod


def _strided(arr, ld):
    """Copy of a 2-D array inside rows of length ``ld``; the padding holds
    NaN (fp32 NaN, or the bf16 quiet-NaN pattern for bf16 bits), so a read of
    it would poison the result."""
    if arr.dtype == np.uint16:
        out = np.full((arr.shape[0], ld), 0x7FC0, dtype=np.uint16)
    else:
        out = np.full((arr.shape[0], ld), np.nan, dtype=np.float32)
    out[:, :arr.shape[1]] = arr
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_random_shapes_instances_and_leading_dims(x, dtype):
    import torch
    rng = np.random.default_rng(20261202 + (dtype == "bf16"))
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    scheds = x.xtc_sched_list(x.XTC_OP_MATMUL, code)
    for case in range(24):
        M, N, K = (int(v) for v in rng.integers(1, 300, size=3))
        pa, pb, pc = (int(v) for v in rng.integers(0, 9, size=3))
        s = scheds[int(rng.integers(len(scheds)))]
        s.raster = int(rng.choice([0, 1, 4, 8]))
        s.xcd_remap = int(rng.integers(2))
        relu = bool(rng.integers(2))
        A = xi.small_int_f32(100 + case, (M, K))
        B = xi.small_int_f32(200 + case, (K, N))
        if dtype == "bf16":
            A, B = xi.f32_to_bf16_bits(A), xi.f32_to_bf16_bits(B)
        ref = oracle.matmul(A, B)
        if relu:
            ref = oracle.relu(ref)
        lda, ldb, ldc = K + pa, N + pb, N + pc
        Ad, Bd = to_dev(_strided(A, lda)), to_dev(_strided(B, ldb))
        Cd = torch.full((M, ldc), 7.0, dtype=torch.float32, device="cuda")
        fn = x.xtc_matmul_relu if relu else x.xtc_matmul
        say("random", dtype, case, (M, N, K), (lda, ldb, ldc), relu, s)
        st = fn(M, N, K, Ad.data_ptr(), lda, Bd.data_ptr(), ldb, Cd.data_ptr(), ldc, code, s,
                torch.cuda.current_stream().cuda_stream)
        assert st == 0, x.xtc_status_str(st)
        got = to_host(Cd)
        assert np.array_equal(got[:, :N], ref), (case, M, N, K, s)
        assert np.all(got[:, N:] == 7.0), "columns past N were written"


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_random_patch_staging_class_convs(x, dtype):
    """Seeded random 3x3 stride-1 layers with rows of about 56 pixels -- the
    class of the kernels that stage an input patch once for all taps
    (k_order 2) -- through every such instance and the default schedule,
    with random raster orders and the fused relu.  Widths, heights, padding,
    channel and output-channel counts vary, so some shapes fall outside a
    kernel's class and exercise its fallback.  Small-integer inputs: every
    result is bit-exact."""
    rng = np.random.default_rng(5656 + (dtype == "bf16"))
    code = x.XTC_F32 if dtype == "f32" else x.XTC_BF16
    scheds = [s for s in x.xtc_sched_list(x.XTC_OP_CONV2D, code) if s.k_order == 2] + [None]
    for case in range(6):
        N = int(rng.integers(1, 3))
        C = int(rng.choice([8, 16, 24, 32, 48]))
        H, W = (int(v) for v in rng.integers(50, 61, size=2))
        OC = int(rng.integers(1, 131))
        pad = int(rng.integers(0, 3))
        relu = bool(rng.integers(2))
        X = xi.small_int_f32(700 + case, (N, C, H, W))
        Wt = xi.small_int_f32(800 + case, (OC, C, 3, 3))
        if dtype == "bf16":
            X, Wt = xi.f32_to_bf16_bits(X), xi.f32_to_bf16_bits(Wt)
        ref = oracle.conv2d(X, Wt, stride=1, pad=pad)
        if relu:
            ref = oracle.relu(ref)
        Xd, Wd = to_dev(X), to_dev(Wt)
        for s in scheds:
            if s is not None:
                s.raster = int(rng.choice([0, 1, 8]))
                s.xcd_remap = int(rng.integers(2))
            say("random conv", dtype, case, (N, C, H, W, OC, pad), relu, s)
            got = to_host(x.conv2d_nchw(Xd, Wd, stride=1, pad=pad, sched=s, relu=relu))
            assert np.array_equal(got, ref), (dtype, case, (N, C, H, W, OC, pad), relu, s)


def test_bf16_rows_at_any_two_byte_boundary(x):
    """bf16 operands whose base pointers sit 1..7 elements past a 16-byte
    boundary, with odd row strides: every row starts at a different 2-byte
    offset, so the register-staged kernels read them with 16-byte loads of
    the covering aligned chunks shifted into place.  Every compiled instance
    and the default schedule, on small integers (bit-exact).  The elements
    around each operand and in the row padding hold the bf16 NaN pattern, so
    a value taken from outside the operand would poison the result."""
    import torch
    rng = np.random.default_rng(97)
    scheds = x.xtc_sched_list(x.XTC_OP_MATMUL, x.XTC_BF16) + [None]
    for case, (M, N, K) in enumerate([(131, 77, 203), (300, 257, 9), (65, 129, 1000)]):
        A = xi.f32_to_bf16_bits(xi.small_int_f32(900 + case, (M, K)))
        B = xi.f32_to_bf16_bits(xi.small_int_f32(950 + case, (K, N)))
        ref = oracle.matmul(A, B)
        lda, ldb = K + int(rng.integers(0, 3)) * 2 + (K % 2 == 0), N + (N % 2 == 0)
        oa, ob = (int(v) for v in rng.integers(1, 8, size=2))

        def place(arr, ld, off):
            rows = arr.shape[0]
            flat = np.full(off + rows * ld + 16, 0x7FC0, dtype=np.uint16)
            flat[off:off + rows * ld] = _strided(arr, ld).ravel()
            return to_dev(flat)

        Ad, Bd = place(A, lda, oa), place(B, ldb, ob)
        pa, pb = Ad.data_ptr() + 2 * oa, Bd.data_ptr() + 2 * ob
        assert pa % 16 and pb % 16
        for s in scheds:
            Cd = torch.full((M, N), 7.0, dtype=torch.float32, device="cuda")
            say("bf16 offset rows", (M, N, K), (lda, ldb), (oa, ob), s)
            st = x.xtc_matmul(M, N, K, pa, lda, pb, ldb, Cd.data_ptr(), N, x.XTC_BF16, s,
                              torch.cuda.current_stream().cuda_stream)
            assert st == 0, x.xtc_status_str(st)
            assert np.array_equal(to_host(Cd), ref), ((M, N, K), (lda, ldb), (oa, ob), s)


def test_random_sweep_every_instance_kind(x):
    """A wider seeded sweep: 240 matmuls (fp32 and bf16, M, N, K up to 700,
    every eighth with at most 32 columns, every eleventh with K up to 3000),
    each through a random compiled instance or the default schedule with a
    random raster order, XCD remap and relu flag, padded leading dimensions,
    NaN around the operands and, for bf16, a base pointer 0-7 elements past a
    16-byte boundary; and 60 convolutions (3x3 stride-1 layers of about 56
    pixels every third case, else small random 1x1/3x3/5x5 layers with
    stride 1 or 2), each through a random instance.  Small-integer inputs:
    every result is bit-exact."""
    import torch
    rng = np.random.default_rng(424242)
    for case in range(240):
        dt = ("f32", "bf16")[case % 2]
        code = x.XTC_F32 if dt == "f32" else x.XTC_BF16
        scheds = x.xtc_sched_list(x.XTC_OP_MATMUL, code) + [None]
        M, N, K = (int(v) for v in rng.integers(1, 700, size=3))
        if case % 8 == 0:
            N = int(rng.integers(1, 33))
        if case % 11 == 0:
            K = int(rng.integers(1, 3000))
        s = scheds[int(rng.integers(len(scheds)))]
        if s is not None:
            s.raster = int(rng.choice([0, 1, 4, 8, 16]))
            s.xcd_remap = int(rng.integers(2))
        pa, pb, pc = (int(v) for v in rng.integers(0, 9, size=3))
        off = int(rng.integers(0, 8)) if dt == "bf16" else 0
        relu = bool(rng.integers(2))
        A = xi.small_int_f32(10000 + case, (M, K))
        B = xi.small_int_f32(20000 + case, (K, N))
        if dt == "bf16":
            A, B = xi.f32_to_bf16_bits(A), xi.f32_to_bf16_bits(B)
        ref = oracle.matmul(A, B)
        if relu:
            ref = oracle.relu(ref)
        lda, ldb, ldc = K + pa, N + pb, N + pc

        def place(arr, ld, o):
            fill = 0x7FC0 if arr.dtype == np.uint16 else np.nan
            flat = np.full(o + arr.shape[0] * ld + 16, fill, dtype=arr.dtype)
            flat[o:o + arr.shape[0] * ld] = _strided(arr, ld).ravel()
            return to_dev(flat)

        Ad, Bd = place(A, lda, off), place(B, ldb, 0)
        Cd = torch.full((M, ldc), 7.0, dtype=torch.float32, device="cuda")
        fn = x.xtc_matmul_relu if relu else x.xtc_matmul
        say("sweep mm", dt, case, (M, N, K), (lda, ldb, ldc), off, relu, s)
        st = fn(M, N, K, Ad.data_ptr() + 2 * off, lda, Bd.data_ptr(), ldb, Cd.data_ptr(), ldc,
                code, s, torch.cuda.current_stream().cuda_stream)
        assert st == 0, x.xtc_status_str(st)
        got = to_host(Cd)
        assert np.array_equal(got[:, :N], ref), (dt, case, (M, N, K), off, relu, s)
        assert np.all(got[:, N:] == 7.0), "columns past N were written"
    for case in range(60):
        dt = ("f32", "bf16")[case % 2]
        code = x.XTC_F32 if dt == "f32" else x.XTC_BF16
        scheds = x.xtc_sched_list(x.XTC_OP_CONV2D, code) + [None]
        n = int(rng.integers(1, 4))
        C = int(rng.choice([3, 8, 16, 24, 32, 48, 64]))
        if case % 3 == 0:
            H, W = (int(v) for v in rng.integers(48, 62, size=2))
            R, stride = 3, 1
        else:
            H, W = (int(v) for v in rng.integers(5, 40, size=2))
            R, stride = int(rng.choice([1, 3, 5])), int(rng.integers(1, 3))
        pad = int(rng.integers(0, 3))
        OC = int(rng.integers(1, 140))
        if H + 2 * pad < R or W + 2 * pad < R:
            continue
        s = scheds[int(rng.integers(len(scheds)))]
        if s is not None:
            s.raster = int(rng.choice([0, 1, 8]))
            s.xcd_remap = int(rng.integers(2))
        relu = bool(rng.integers(2))
        X = xi.small_int_f32(30000 + case, (n, C, H, W))
        Wt = xi.small_int_f32(40000 + case, (OC, C, R, R))
        if dt == "bf16":
            X, Wt = xi.f32_to_bf16_bits(X), xi.f32_to_bf16_bits(Wt)
        ref = oracle.conv2d(X, Wt, stride=stride, pad=pad)
        if relu:
            ref = oracle.relu(ref)
        say("sweep conv", dt, case, (n, C, H, W, OC, R, stride, pad), relu, s)
        got = to_host(x.conv2d_nchw(to_dev(X), to_dev(Wt), stride=stride, pad=pad, sched=s, relu=relu))
        assert np.array_equal(got, ref), (dt, case, (n, C, H, W, OC, R, stride, pad), relu, s)


def test_concurrent_host_threads_on_separate_streams(x):
    import torch
    jobs = []
    for t in range(4):
        M, N, K = 200 + 37 * t, 150 + 19 * t, 300 + 11 * t
        jobs.append(("mm", xi.small_int_f32(300 + t, (M, K)), xi.small_int_f32(400 + t, (K, N))))
    jobs.append(("conv", xi.small_int_f32(500, (2, 16, 20, 22)), xi.small_int_f32(501, (24, 16, 3, 3))))
    jobs.append(("bf16", xi.f32_to_bf16_bits(xi.small_int_f32(600, (333, 129))),
                 xi.f32_to_bf16_bits(xi.small_int_f32(601, (129, 257)))))
    refs = []
    for kind, a, b in jobs:
        if kind == "conv":
            refs.append(oracle.conv2d(a, b, stride=1, pad=1))
        else:
            refs.append(oracle.relu(oracle.matmul(a, b)) if kind == "mm" else oracle.matmul(a, b))
    results = [None] * len(jobs)
    errors = []

    def worker(i):
        try:
            stream = torch.cuda.Stream()
            kind, a, b = jobs[i]
            with torch.cuda.stream(stream):
                ad, bd = to_dev(a), to_dev(b)
                outs = []
                for _ in range(5):   # repeated launches overlap with the other threads'
                    if kind == "conv":
                        outs.append(x.conv2d_nchw(ad, bd, stride=1, pad=1))
                    else:
                        outs.append(x.matmul(ad, bd, relu=(kind == "mm")))
                stream.synchronize()
                results[i] = [o.cpu().numpy() for o in outs]
        except Exception as e:  # reported by the main thread
            errors.append(repr(e))

    say("concurrent", len(jobs), "threads")
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(jobs))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    for i, ref in enumerate(refs):
        assert results[i] is not None
        for got in results[i]:
            assert np.array_equal(got, ref), "job %d" % i
