"""Property tests of the host-side validation in libxtc.so (no GPU needed):
arbitrary schedule fields and shapes never crash the checks, every answer is
one of the documented status codes, a schedule the check accepts is one of
the compiled instances, and invalid calls are refused before any device
work (dummy pointers that a kernel would fault on)."""
import pytest
from hypothesis import HealthCheck, example, given, settings
from hypothesis import strategies as st

I32 = st.one_of(st.integers(-2 ** 31, 2 ** 31 - 1), st.sampled_from([0, 1, 2, 4, 8, 16, 32, 64, 128, 256, 512, -1]))
FIELDS = ("block_m", "block_n", "block_k", "wave_m", "wave_n", "mfma_m", "mfma_n", "mfma_k",
          "lds_stages", "lds_pad", "unroll_k", "raster", "xcd_remap", "k_order", "k_split")


@pytest.fixture(scope="module")
def x():
    import paper_2512_16512_amd as mod
    return mod


@settings(max_examples=400, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(vals=st.fixed_dictionaries({f: I32 for f in FIELDS}), op=st.sampled_from([0, 1]),
       dt=st.sampled_from([0, 1]))
def test_sched_check_total_and_sound(x, vals, op, dt):
    s = x.Sched(**vals)
    st_ = x.xtc_sched_check(op, dt, s)
    assert st_ in (0, 4, 5, 6)
    if st_ == 0:
        keys = {tuple(sorted(c.as_dict().items())) for c in x.xtc_sched_list(op, dt)}
        d = s.as_dict()
        d["raster"], d["xcd_remap"] = 0, 1
        assert tuple(sorted(d.items())) in keys


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(M=st.integers(-5, 2 ** 63 - 1), N=st.integers(-5, 2 ** 63 - 1), K=st.integers(-5, 2 ** 63 - 1),
       pads=st.tuples(*[st.one_of(st.just(0), st.integers(0, 2 ** 63 - 1))] * 3),
       dt=st.sampled_from([0, 1]))
@example(M=(1 << 62) + 1, N=4, K=4, pads=(0, 0, 0), dt=0)   # (M - 1) * ld wraps to 0
def test_huge_or_negative_shapes_refused_before_launch(x, M, N, K, pads, dt):
    # leading dimensions at least the extents, up to 2^63 - 1 (products of
    # such sizes overflow 64 bits); pointers are dummies, so only the no-op
    # (M or N == 0) or a refusal may come back
    BAD = 0x10
    lim = 2 ** 63 - 1
    lda, ldb, ldc = (min(max(e, 1) + p, lim) for e, p in zip((K, N, N), pads))
    # Only calls that are clearly invalid are made: negative or zero extents,
    # or an operand span of at least twice the 2^31-byte limit.  Anything
    # near the limit is skipped, so that no call can reach a launch on the
    # dummy pointers.
    spans = [(max(M, 1) - 1) * lda + K, (max(K, 1) - 1) * ldb + N, (max(M, 1) - 1) * ldc + N]
    clearly_large = max(spans) * 2 >= 2 ** 32
    if not (M < 0 or N < 0 or K < 0 or M == 0 or N == 0 or clearly_large):
        return
    st_ = x.xtc_matmul(M, N, K, BAD, lda, BAD, ldb, BAD, ldc, dt)
    assert st_ in (0, 2, 3, 7)
    if M < 0 or N < 0 or K < 0:
        assert st_ == 2
    elif M == 0 or N == 0:
        assert st_ == 0
    else:
        assert st_ == 7   # an operand span past the limit, however large


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(op=st.sampled_from([0, 1]), dt=st.sampled_from([0, 1]),
       M=st.one_of(st.integers(0, 1 << 20), st.integers(0, 2 ** 63 - 1)),
       N=st.one_of(st.integers(0, 1 << 24), st.integers(0, 2 ** 63 - 1)),
       K=st.one_of(st.integers(0, 1 << 16), st.integers(0, 2 ** 63 - 1)))
def test_default_schedule_is_always_compiled(x, op, dt, M, N, K):
    s = x.xtc_default_schedule(op, dt, M, N, K)
    assert x.xtc_sched_check(op, dt, s) == 0


SIZE = st.one_of(st.integers(-2, 9), st.integers(-2, 2 ** 63 - 1))


@settings(max_examples=400, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])
@given(dims=st.tuples(*[SIZE] * 11), dt=st.sampled_from([0, 1]))
@example(dims=(1 << 61, 1, 4, 4, 1, 3, 3, 1, 1, 0, 0), dt=0)   # X and Y spans wrap to 0
@example(dims=(1, 1 << 62, 4, 4, 1, 3, 3, 1, 1, 0, 0), dt=1)   # C * R * S wraps
def test_conv_invalid_or_huge_refused_before_launch(x, dims, dt):
    # The conv checks in their order: shape signs, strides / pads / padded
    # extents above 2^30, a kernel larger than the padded input, the no-op
    # (N or OC == 0), then the operand spans (2^31-byte limit).  Pointers
    # are dummies, so only calls that one of these decides are made: a
    # valid call of modest size is skipped (it would launch).
    N, C, H, W, OC, R, S, sh, sw, ph, pw = dims
    BAD = 0x10
    lim = 2 ** 30
    if (N < 0 or OC < 0 or C < 1 or H < 1 or W < 1 or R < 1 or S < 1 or sh < 1 or sw < 1
            or ph < 0 or pw < 0):
        expected = 2
    elif max(sh, sw, ph, pw, H, W) > lim or H + 2 * ph > lim or W + 2 * pw > lim:
        expected = 7
    elif H + 2 * ph < R or W + 2 * pw < S:
        expected = 2
    elif N == 0 or OC == 0:
        expected = 0
    else:
        OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
        elt = 4 if dt == 0 else 2
        spans = [N * C * H * W * elt, OC * C * R * S * elt, N * OC * OH * OW * 4]
        if max(spans) * 2 < 2 ** 32:
            return
        expected = 7
    assert x.xtc_conv2d_nchw(N, C, H, W, OC, R, S, sh, sw, ph, pw, BAD, BAD, BAD, dt) == expected
