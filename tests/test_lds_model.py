"""CPU tests of the LDS bank-conflict model (paper_2512_16512_amd/lds_model.py).

The model's predictions are pinned to counter values rocprofv3 measured on
MI355X (SQ_LDS_IDX_ACTIVE, SQ_LDS_BANK_CONFLICT per dispatch; the profiles
under profiles/ hold the commands), and its phase tables to the probe
measurements that define them.
"""
import pytest

from paper_2512_16512_amd import lds_model as L


def _frag_modes(mode):
    """Lane byte addresses of the ds_read_b128 patterns a throughput probe
    measured at 4, 8, 16 and 16 LDS cycles per instruction."""
    out = []
    for lane in range(64):
        row, g = lane & 31, lane >> 5
        if mode == 0:
            out.append(16 * lane)
        elif mode == 1:
            out.append(row * 64 + ((g ^ ((row >> 1) ^ (row >> 3))) & 3) * 16)
        elif mode == 2:
            out.append(row * 64 + ((g + row) & 3) * 16)
        else:
            out.append(row * 64 + ((g ^ (row & 3)) & 3) * 16)
    return out


def test_phase_tables_reproduce_probe_cycles():
    assert [L.cycles("ds_read_b128", _frag_modes(m)) for m in range(4)] == [4, 8, 16, 16]


def test_phase_tables_partition_the_wave():
    for op, phases in L.PHASES.items():
        lanes = sorted(l for p in phases for l in p)
        assert lanes == list(range(64)), op


def test_contiguous_accesses_are_conflict_free():
    for op, w in L.WIDTH.items():
        addrs = [w * lane for lane in range(64)]
        assert L.cycles(op, addrs) == L.ideal(op), op


def test_bank_periods():
    # two lanes of one phase, same bank at the measured period, else distinct
    for op, period in (("ds_read_b32", 128), ("ds_write_b128", 128), ("ds_read_b128", 256),
                       ("ds_read_b64_tr_b16", 256)):
        base = [None] * 64
        a = list(base)
        a[0], a[1] = 0, period
        assert L.cycles(op, a) == 2, op
        a[1] = period // 2 if op != "ds_read_b32" else 64
        assert L.cycles(op, a) == 1, op


# (prediction, measured SQ_LDS_IDX_ACTIVE, measured SQ_LDS_BANK_CONFLICT)
BF16_8192 = dict(block_m=256, block_n=256, block_k=32, wave_m=128, wave_n=64, mfma_m=32,
                 lds_pad=-1, k_split=1)


def test_bf16_gemm_8192_matches_counters():
    c = L.matmul_launch("bf16", BF16_8192, 8192, 8192, 8192)
    assert c.active == pytest.approx(1.009e8, rel=2e-3) and c.conflict == 0


def test_bf16_gemm_previous_swizzle_matches_counters():
    old = lambda ca, row: ((row >> 1) ^ (row >> 3)) & 3 if ca == 4 else (row ^ (row >> 3)) & 7
    c = L.gemm_bf16_dma_launch(BF16_8192, 8192, 8192, 8192, swz_a=old)
    assert c.active == pytest.approx(1.681e8, rel=2e-3)
    assert c.conflict == pytest.approx(6.724e7, rel=2e-3)


def test_f32_gemm_4096_matches_counters():
    s = dict(block_m=256, block_n=256, block_k=32, wave_m=128, wave_n=64, mfma_m=32, lds_pad=-1,
             k_split=1)
    c = L.matmul_launch("f32", s, 4096, 4096, 4096)
    assert c.active == pytest.approx(3.362e7, rel=2e-3) and c.conflict == 0


def test_ksplit_reduction_matches_counters():
    s = dict(block_m=32, block_n=16, block_k=32, wave_m=32, wave_n=16, mfma_m=16, lds_pad=0,
             k_split=8)
    c = L.matmul_launch("f32", s, 32768, 16, 4096)
    assert c.active == 262144 and c.conflict == 0


def test_f32_halo_conv_matches_counters_before_and_after():
    before = L.conv_f32_halo16_launch(32, 64, 56, 56, 64, 1, 1, plane_pad=16, a_swizzle=False)
    assert before.active == pytest.approx(1.0617e7, rel=2e-3)
    assert before.conflict == pytest.approx(2.654e6, rel=2e-3)
    # a layout measured on the way (planes 32 floats apart, channels 8..15 at c ^ 2)
    wrong = L.conv_f32_halo16_launch(32, 64, 56, 56, 64, 1, 1, plane_pad=32,
                                     a_swizzle=lambda lcol: ((lcol >> 3) & 1) << 1)
    assert wrong.active == pytest.approx(1.593e7, rel=2e-3)
    assert wrong.conflict == pytest.approx(7.963e6, rel=2e-3)
    now = L.conv_launch("f32", dict(k_order=2, block_n=416, block_m=64, lds_stages=2),
                        32, 64, 56, 56, 64, 3, 3, 1, 1)
    assert now.active == pytest.approx(8.847e6, rel=2e-3)
    assert now.conflict == pytest.approx(8.847e5, rel=2e-3)


def test_bf16_halo_conv_matches_counters():
    # the kernel before its bank layouts (and before its loads went two
    # stages ahead, when the last stage still stored a next one)
    old = L.conv_bf16_halo_launch(32, 64, 56, 56, 64, 1, 1, trailing_store=True)
    assert old.active == pytest.approx(2.463e6, rel=0.02)
    assert old.conflict == pytest.approx(9.39e5, rel=0.06)
    # the current kernel: SQ_LDS_IDX_ACTIVE 1411072 and 40704 per launch on
    # the two shapes, no conflicts
    now = L.conv_launch("bf16", dict(k_order=2, block_n=256, block_m=64, lds_stages=2),
                        32, 64, 56, 56, 64, 3, 3, 1, 1)
    assert now.active == 1411072 and now.conflict == 0
    small = L.conv_launch("bf16", dict(k_order=2, block_n=256, block_m=64, lds_stages=2),
                          3, 64, 13, 54, 16, 3, 3, 1, 2)
    assert small.active == 40704 and small.conflict == 0


def test_bf16_row_streaming_conv_matches_counters():
    # SQ_LDS_IDX_ACTIVE per launch of the row-streaming kernel (k_order 3,
    # output rows staged through LDS for the stores, bands of whole steps),
    # measured: 1874432 and 67200 cycles on the two shapes, no conflicts
    s = dict(k_order=3, block_n=64, block_m=64, lds_stages=2)
    c = L.conv_launch("bf16", s, 32, 64, 56, 56, 64, 3, 3, 1, 1)
    assert c.active == 1874432 and c.conflict == 0
    c = L.conv_launch("bf16", s, 3, 64, 13, 54, 16, 3, 3, 1, 2)
    assert c.active == 67200 and c.conflict == 0
    # outside its class the launcher runs the halo kernel, and so does the model
    h = L.conv_launch("bf16", s, 1, 48, 56, 58, 16, 3, 3, 1, 2)
    assert h is not None and h.active == L.conv_launch(
        "bf16", dict(k_order=2, block_n=256, block_m=64, lds_stages=2), 1, 48, 56, 58, 16, 3, 3, 1, 2).active


def test_small_channel_conv_matches_counters():
    # measured on the patch-staged kernel with two reduction halves and
    # 16-byte patch rows: 279888 LDS-active cycles and 8624 conflict cycles
    # per launch (7x7 layer), 373184 and 18816 (4x16x56x56 -> 16, 3x3)
    s = dict(k_order=0, block_n=64, block_m=16, lds_stages=0)
    c = L.conv_launch("f32", s, 1, 3, 224, 224, 16, 7, 7, 2, 3)
    assert c.active == pytest.approx(279888, rel=1e-2)
    assert c.conflict == 8624
    c = L.conv_launch("f32", s, 4, 16, 56, 56, 16, 3, 3, 1, 1)
    assert c.active == pytest.approx(373184, rel=1e-2)
    assert c.conflict == 18816


def test_f32_64x256_halo_conv_matches_counters():
    # measured SQ_LDS_IDX_ACTIVE / SQ_LDS_BANK_CONFLICT per launch, with
    # conflicts (this kernel is not a default): 4672000 / 1756672 and
    # 152000 / 57152
    s = dict(k_order=2, block_m=64, block_n=256, block_k=8, wave_m=64, wave_n=64, mfma_m=32,
             lds_stages=2, lds_pad=-1)
    c = L.conv_launch("f32", s, 32, 64, 56, 56, 64, 3, 3, 1, 1)
    assert (c.active, c.conflict) == (4672000, 1756672)
    c = L.conv_launch("f32", s, 4, 16, 56, 56, 16, 3, 3, 1, 1)
    assert (c.active, c.conflict) == (152000, 57152)
    # outside its class the launcher falls back to the tap-major kernel
    assert L.conv_launch("f32", s, 8, 128, 28, 28, 256, 3, 3, 1, 1).active == 1382400
    # the few-channel kernel's gather form (the patch does not fit) is not modelled
    few = dict(k_order=0, block_m=16, block_n=64, lds_stages=0)
    assert L.conv_launch("f32", few, 32, 64, 56, 56, 64, 3, 3, 1, 1) is None


def _conv_inst(bm, bn, wm, wn, mi, stages, pad, k_order, bk=32):
    return dict(block_m=bm, block_n=bn, block_k=bk, wave_m=wm, wave_n=wn, mfma_m=mi,
                lds_stages=stages, lds_pad=pad, k_order=k_order)


# SQ_LDS_IDX_ACTIVE and SQ_LDS_BANK_CONFLICT per launch, measured (mean of
# two launches, equal): the fp32 gather conv kernels as the launchers chain
# them (tap-major for C % 32 == 0, else the k-table direct-to-LDS kernel with
# the fallback's stages, else the register-staged kernel)
MEASURED_GATHER = [
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(64, 128, 32, 64, 32, 2, -1, 1), 4515840, 0),
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(128, 128, 64, 64, 32, 3, -1, 0), 6500928, 0),
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(64, 128, 32, 64, 16, 2, 4, 0), 11769408, 903168),
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(128, 128, 64, 64, 32, 2, 4, 0), 12672576, 0),
    ((8, 128, 28, 28, 256, 3, 3, 1, 1), _conv_inst(128, 128, 64, 64, 32, 2, -1, 1), 1354752, 0),
    ((4, 16, 56, 56, 16, 3, 3, 1, 1), _conv_inst(64, 256, 64, 64, 32, 2, -1, 1), 116620, 0),
    ((4, 16, 56, 56, 16, 3, 3, 1, 1), _conv_inst(64, 128, 32, 64, 32, 2, 4, 0), 364952, 0),
    ((2, 24, 30, 30, 40, 5, 5, 2, 2), _conv_inst(64, 128, 32, 64, 32, 3, -1, 0), 30112, 0),
    ((2, 24, 30, 30, 40, 5, 5, 2, 2), _conv_inst(128, 128, 64, 64, 32, 2, -1, 1), 34976, 0),
]


@pytest.mark.parametrize("dims,s,active,conflict", MEASURED_GATHER)
def test_gather_conv_kernels_match_counters(dims, s, active, conflict):
    c = L.conv_launch("f32", s, *dims)
    assert c.active == active and c.conflict == conflict


def test_gather_conv_fallbacks_match_counters():
    # C*R*S = 147 and 45 are not multiples of 4: every gather instance runs
    # the register-staged kernel (measured 367010 and 11074 for 64x128 tiles)
    for dims, meas in (((1, 3, 224, 224, 16, 7, 7, 2, 3), 367010), ((3, 5, 17, 19, 33, 3, 3, 1, 1), 11074)):
        for s in (_conv_inst(64, 128, 32, 64, 32, 2, -1, 1), _conv_inst(64, 128, 32, 64, 32, 3, -1, 0),
                  _conv_inst(64, 128, 32, 64, 32, 2, 4, 0)):
            assert L.conv_launch("f32", s, *dims).active == meas
    # the 64x64 k-table tile: the compiler skips one table read per stage
    # past the end of K, which the model counts (measured 7545216)
    c = L.conv_launch("f32", _conv_inst(64, 64, 32, 32, 32, 3, -1, 0), 32, 64, 56, 56, 64, 3, 3, 1, 1)
    assert 1.0 < c.active / 7545216 < 1.01


def test_tap_major_is_the_fragment_reads_only():
    # no table: K-stages x four fragment sets of the direct-to-LDS GEMM's
    # reads (with the conv's weight swizzle) per workgroup
    s = _conv_inst(64, 128, 32, 64, 32, 2, -1, 1)
    c = L.conv_launch("f32", s, 32, 64, 56, 56, 64, 3, 3, 1, 1)
    stage = L.gemm_f32_dma_stage(64, 128, 32, 32, 64, 32, swz_a=lambda ca, row: (row ^ (row >> 3)) & 7)
    assert c.active == stage.active * (576 // 32) * (32 * 56 * 56 // 128)


def test_staged_k_split_matches_counters():
    # the fp32 direct-to-LDS kernel in two and four K groups on 1000^3:
    # SQ_LDS_IDX_ACTIVE 1662976 and 1818624 per launch (unsplit: 1585152),
    # no conflicts
    base = dict(block_m=64, block_n=64, block_k=32, wave_m=32, wave_n=32, mfma_m=32,
                lds_stages=2, lds_pad=-1)
    for ks, cyc in ((1, 1585152), (2, 1662976), (4, 1818624)):
        c = L.matmul_launch("f32", dict(base, k_split=ks), 1000, 1000, 1000)
        assert c.active == cyc and c.conflict == 0


# bf16 gather kernel (k_order 0, the halo kernel's fallback): measured
# SQ_LDS_IDX_ACTIVE / SQ_LDS_BANK_CONFLICT per launch, equal to the model
MEASURED_BF16_GATHER = [
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(64, 128, 32, 64, 32, 2, 8, 0), 7705152, 451584),
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(64, 128, 32, 64, 16, 2, 8, 0, bk=64), 8608320, 1354752),
    ((32, 64, 56, 56, 64, 3, 3, 1, 1), _conv_inst(64, 128, 32, 64, 32, 2, 8, 0, bk=64), 7253568, 0),
    ((3, 64, 13, 54, 16, 3, 3, 1, 2), _conv_inst(64, 64, 32, 32, 32, 2, 8, 0), 228384, 23040),
    ((3, 64, 13, 54, 16, 3, 3, 1, 2), _conv_inst(128, 128, 64, 64, 32, 2, 8, 0), 227664, 23040),
]


@pytest.mark.parametrize("dims,s,active,conflict", MEASURED_BF16_GATHER)
def test_bf16_gather_conv_matches_counters(dims, s, active, conflict):
    c = L.conv_launch("bf16", s, *dims)
    assert c.active == active and c.conflict == conflict


def test_register_staged_table_reads_follow_the_padding():
    # the second word of a table entry is read only when the tap falls in the
    # image for one of the wave's pixels: every 3x3 tap does on 56x56 images,
    # so both words are read for every gathered row (2 x N*OH*OW*K/64 reads),
    # while with padding 2 on 13 rows some taps leave whole waves outside
    full = L._reg_table_reads(32, 64, 56, 56, 3, 3, 1, 1, 1, 1, 128, 4, 32)
    assert full == 2 * 32 * 56 * 56 * 576 // 64
    padded = L._reg_table_reads(3, 64, 13, 54, 3, 3, 1, 1, 2, 2, 128, 4, 32)
    assert padded < 2 * 3 * 15 * 56 * 576 // 64 + 4 * 576


def test_register_staged_fp32_conv_exact_on_five_shapes():
    # 64x128 tiles, 32x32x2 instructions, rows padded by 4 floats: measured
    for dims, meas in (((32, 64, 56, 56, 64, 3, 3, 1, 1), 10866240), ((4, 16, 56, 56, 16, 3, 3, 1, 1), 364952),
                       ((1, 3, 224, 224, 16, 7, 7, 2, 3), 367010), ((3, 5, 17, 19, 33, 3, 3, 1, 1), 11074),
                       ((2, 24, 30, 30, 40, 5, 5, 2, 2), 58032)):
        assert L.conv_launch("f32", _conv_inst(64, 128, 32, 64, 32, 2, 4, 0), *dims).active == meas
