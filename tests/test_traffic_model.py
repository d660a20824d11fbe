"""The analytic HBM-traffic model (paper_2512_16512_amd.traffic_model) on the
CPU: its tile map, closed forms of its prediction, its correlation statistics
against scipy, and the matching of profiler rows to schedules."""
import csv
import json
import random

import numpy as np
import pytest
import scipy.stats

from paper_2512_16512_amd import traffic_model as tm


@pytest.mark.parametrize("tiles_m,tiles_n", [(1, 1), (3, 5), (8, 8), (13, 7), (32, 32), (5, 40)])
@pytest.mark.parametrize("raster,xcd", [(0, 0), (0, 1), (1, 0), (1, 1), (4, 1), (8, 0), (16, 1)])
def test_tile_map_is_a_bijection(tiles_m, tiles_n, raster, xcd):
    g = tiles_m * tiles_n
    seen = {tm.tile_coords(b, g, tiles_m, tiles_n, raster, xcd) for b in range(g)}
    assert seen == {(i, j) for i in range(tiles_m) for j in range(tiles_n)}


def test_single_tile_reads_both_operands_once():
    r, w = tm.predict(100, 70, 300, 4, 128, 128, 0, 1, 1)
    assert r == (100 + 70) * 300 * 4 and w == 4 * 100 * 70


def test_one_tile_per_xcd_reads_every_panel_per_tile():
    # 2 x 4 = 8 tiles: each XCD holds one tile, so nothing is shared
    M, N, K = 64 * 2, 32 * 4, 50
    r, _ = tm.predict(M, N, K, 2, 64, 32, 0, 0, 1, l2_bytes=0)
    assert r == 8 * (64 + 32) * K * 2


def test_everything_resident_reads_each_panel_once_per_xcd():
    M, N, K, bm, bn = 1024, 1024, 64, 64, 64
    r, _ = tm.predict(M, N, K, 4, bm, bn, 0, 0, 1, l2_bytes=1 << 40)
    tiles_m = tiles_n = 16
    expect = 0
    for x in range(8):
        ts = [tm.tile_coords(b, 256, tiles_m, tiles_n, 0, 0) for b in range(x, 256, 8)]
        expect += (len({t[0] for t in ts}) * bm + len({t[1] for t in ts}) * bn) * K * 4
    assert r == expect
    # row-major without remap: XCD x gets columns x and x+8 of every row
    assert r == 8 * (16 * 64 + 2 * 64) * K * 4


def test_streaming_regime_counts_groups():
    # one XCD band per group: with the remap and row-major raster, XCD x gets
    # 32 consecutive tiles = one tile-row of 32 tiles, one group at occupancy 1
    M, N, K = 8 * 128, 32 * 128, 4096
    r, _ = tm.predict(M, N, K, 4, 128, 128, 0, 1, 1, l2_bytes=0)
    assert r == 8 * (1 * 128 + 32 * 128) * K * 4
    # without the remap XCD x gets every 8th tile: 4 tiles of each row
    r0, _ = tm.predict(M, N, K, 4, 128, 128, 0, 0, 1, l2_bytes=0)
    assert r0 == 8 * (8 * 128 + 4 * 128) * K * 4
    assert r0 < r   # a square-ish footprint shares more than one tile-row


def test_ragged_edges_count_real_rows():
    r, _ = tm.predict(130, 10, 7, 4, 128, 128, 0, 1, 1, l2_bytes=0)
    assert r == ((128 + 10) + (2 + 10)) * 7 * 4


def test_correlation_statistics_match_scipy():
    rng = random.Random(5)
    x = [rng.randint(0, 20) for _ in range(60)]          # ties on purpose
    y = [v * 0.5 + rng.random() * 4 for v in x]
    assert abs(tm.pearson(x, y) - scipy.stats.pearsonr(x, y)[0]) < 1e-12
    assert abs(tm.spearman(x, y) - scipy.stats.spearmanr(x, y)[0]) < 1e-12


def test_correlate_matches_rows_to_schedules(tmp_path):
    scheds = [dict(block_m=128, block_n=128, raster=r, xcd_remap=1) for r in (0, 8)]
    order = {"dtype": "f32", "M": 1024, "N": 1024, "K": 1024, "reps": 2,
             "schedules": [{"sched": s, "occupancy": 1} for s in scheds]}
    op = tmp_path / "order.json"
    op.write_text(json.dumps(order))
    cp = tmp_path / "c.csv"
    with open(cp, "w", newline="") as f:
        w = csv.writer(f)
        w.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        did = 0
        for i, v in enumerate([10, 12, 20, 22]):
            w.writerow([did, "void at::native::fill", "FETCH_SIZE", 999]); did += 1
            w.writerow([did, "void xtc::(anonymous namespace)::gemm", "FETCH_SIZE", v]); did += 1
    table, r, rho = tm.correlate(str(op), str(cp), 2.0)
    assert [t["measured"] for t in table] == [11 * 1024 * 2.0, 21 * 1024 * 2.0]
    assert table[0]["predicted"] == tm.predict(1024, 1024, 1024, 4, 128, 128, 0, 1, 1)[0]
    # both schedules fit the same resident footprint: a constant prediction
    assert table[0]["predicted"] == table[1]["predicted"]
    assert r != r and rho != rho          # NaN: correlation undefined


# ---------------------------------------------------- DRAM behind the MALL


def test_dram_is_compulsory_when_operands_fit_the_mall():
    # 8192^3 bf16: A and B are 256 MiB, the MALL's size; every order reads them once
    for raster in (0, 1, 4, 8):
        for xcd in (0, 1):
            d = tm.predict_dram(8192, 8192, 8192, 2, 256, 256, raster, xcd, 1)
            assert d == 2 * 8192 * 8192 * 2


def test_dram_between_compulsory_and_l2_misses():
    M, N, K = 16384, 16384, 8192
    for raster in (0, 1, 2, 4, 8, 16, 32):
        for xcd in (0, 1):
            d = tm.predict_dram(M, N, K, 2, 256, 256, raster, xcd, 1)
            l2, _ = tm.predict(M, N, K, 2, 256, 256, raster, xcd, 1)
            assert (M + N) * K * 2 <= d <= l2


def test_dram_falls_with_a_larger_last_level_cache():
    M, N, K = 16384, 16384, 8192
    small = tm.predict_dram(M, N, K, 2, 256, 256, 0, 0, 1, mall_bytes=64 << 20)
    mid = tm.predict_dram(M, N, K, 2, 256, 256, 0, 0, 1, mall_bytes=256 << 20)
    huge = tm.predict_dram(M, N, K, 2, 256, 256, 0, 0, 1, mall_bytes=4 << 30)
    assert small >= mid >= huge == (M + N) * K * 2


# ---------------------------------------------------------------- conv model

def _sched(**kw):
    d = dict(block_m=64, block_n=128, block_k=32, wave_m=32, wave_n=64, mfma_m=32, mfma_n=32,
             mfma_k=2, lds_stages=3, lds_pad=-1, unroll_k=0, raster=0, xcd_remap=1, k_order=0, k_split=1)
    d.update(kw)
    return d


def test_conv_one_image_per_xcd_reads_input_once():
    # 8 images of 16x16 (one 64x256 flattened tile each), XCD remap: each XCD
    # reads exactly one image and the weights of the one output-channel tile
    dims = (8, 32, 16, 16, 64, 3, 3, 1, 1)
    r, w = tm.predict_conv("f32", _sched(block_n=256), dims, 1)
    assert r == 8 * 32 * 16 * 16 * 4 + 8 * 64 * 32 * 9 * 4
    assert w == 8 * 64 * 16 * 16 * 4


def test_conv_halo_rows_are_read_by_both_neighbouring_xcds():
    # one 32x32 image cut into 8 flattened tiles of 4 output rows: with
    # round-robin XCDs every tile sits on its own XCD and reads its 4 rows
    # plus the rows above and below it (3x3, pad 1), clipped at the image edge
    N, C, H, W = 1, 16, 32, 32
    dims = (N, C, H, W, 64, 3, 3, 1, 1)
    r, _ = tm.predict_conv("f32", _sched(block_n=128, xcd_remap=0), dims, 1)
    rows = sum(min(H - 1, 4 * t + 4) - max(0, 4 * t - 1) + 1 for t in range(8))
    assert rows == 8 * 6 - 2
    assert r == rows * C * W * 4 + 8 * 64 * C * 9 * 4


def test_conv_grid_follows_the_launchers():
    # the benchmark layer: balanced halo tiles of 196 (one half) or 392
    # pixels (two halves), row-streaming bands of 8 rows (whole two-row
    # steps, 7 per image) for bf16
    dims = (32, 64, 56, 56, 64, 3, 3, 1, 1)
    bm, tmm, tn, seg, force = tm.conv_grid("f32", _sched(block_n=208, k_order=2, block_k=8), *dims)
    assert (bm, tmm, tn, force) == (64, 1, 32 * 16, None)
    assert seg(17) == [(1, 2, 7)]             # image 1, pixels 196..391: output rows 3..6
    bm, tmm, tn, seg, force = tm.conv_grid("f32", _sched(block_n=416, k_order=2, block_k=8), *dims)
    assert tn == 32 * 8
    bm, tmm, tn, seg, force = tm.conv_grid("bf16", _sched(block_n=64, k_order=3), *dims)
    assert (tn, force) == (32 * 7, 1) and seg(8) == [(1, 7, 16)]   # band 1: input rows 7 .. 16
    assert seg(6) == [(0, 47, 55)]            # last band: input rows 47 .. 55, row 56 is padding
    # 28x28 rows are too short for the halo tiles: the tap-major 64x256
    # fallback, whose flattened tiles run across images
    small = (8, 128, 28, 28, 256, 3, 3, 1, 1)
    bm, tmm, tn, seg, force = tm.conv_grid("f32", _sched(block_n=208, k_order=2, block_k=8), *small)
    assert (bm, tmm, tn) == (64, 4, -(-8 * 784 // 256))
    assert seg(3) == [(0, 26, 27), (1, 0, 9)]   # pixels 768..1023 span images 0 and 1
    # bf16 with 128 channels: no row streaming, no halo tile; the gather kernel's 64x128 tiles
    bm, tmm, tn, seg, force = tm.conv_grid("bf16", _sched(block_n=64, k_order=3), *small)
    assert (bm, tn) == (64, 8 * 784 // 128)


# FETCH_SIZE x 1024 x 1.9998 bytes per launch (mean of two), one counter pass
# per shape: (dtype, dims, instance fields, raster, remap, occupancy) -> bytes
MEASURED_CONV = [
    ("f32", (32, 64, 56, 56, 64, 3, 3, 1, 1), dict(block_n=416, block_k=8, k_order=2, lds_stages=2), 0, 1, 1, 28.06e6),
    ("f32", (32, 64, 56, 56, 64, 3, 3, 1, 1), dict(block_n=256, k_order=1, lds_stages=2), 0, 1, 2, 27.70e6),
    ("f32", (8, 128, 28, 28, 256, 3, 3, 1, 1), dict(block_n=128, k_order=1, lds_stages=2), 0, 0, 3, 24.59e6),
    ("f32", (8, 128, 28, 28, 256, 3, 3, 1, 1), dict(block_n=64, k_order=1, lds_stages=2), 1, 0, 5, 28.22e6),
    ("f32", (8, 128, 28, 28, 256, 3, 3, 1, 1), dict(block_m=128, block_n=128, k_order=1, lds_stages=2), 0, 1, 2, 12.32e6),
    ("bf16", (32, 64, 56, 56, 64, 3, 3, 1, 1), dict(block_n=64, block_k=16, k_order=3, lds_stages=2), 0, 0, 1, 13.64e6),
    ("bf16", (8, 128, 28, 28, 256, 3, 3, 1, 1), dict(block_n=64, k_order=0, lds_stages=2), 0, 0, 5, 17.68e6),
]


@pytest.mark.parametrize("dtype,dims,fields,raster,remap,occ,measured", MEASURED_CONV)
def test_conv_model_against_counters(dtype, dims, fields, raster, remap, occ, measured):
    r, _ = tm.predict_conv(dtype, _sched(raster=raster, xcd_remap=remap, **fields), dims, occ)
    assert 0.9 <= r / measured <= 1.0


# ------------------------------------------------ L2 reads (the CU side)


def _l2_brute(M, N, K, elt, bm, bn, bk, keep):
    """Lines (A and B kept apart) of every in-range element a tile reads,
    per stage, or per tile when lines survive from stage to stage: sets of
    line numbers, one element at a time."""
    total = 0
    for tm_ in range(-(-M // bm)):
        for tn in range(-(-N // bn)):
            ms = range(tm_ * bm, min(M, (tm_ + 1) * bm))
            ns = range(tn * bn, min(N, (tn + 1) * bn))
            groups = [range(0, K)] if keep else [range(k0, min(K, k0 + bk)) for k0 in range(0, K, bk)]
            for ks in groups:
                a = {(m * K + k) * elt // 128 for m in ms for k in ks}
                b = {(k * N + n) * elt // 128 for k in ks for n in ns}
                total += len(a) + len(b)
    return total * 128


@pytest.mark.parametrize("M,N,K,elt,bm,bn,bk", [
    (5, 24, 40, 4, 4, 16, 8),       # 160-byte rows: runs straddle lines
    (7, 40, 33, 2, 4, 16, 16),      # ragged K and N, bf16
    (16, 16, 64, 4, 8, 8, 16),      # 64-byte B rows: neighbouring rows share a line
    (3, 100, 24, 4, 2, 32, 4),      # 16-byte A runs, ragged column tile
])
def test_l2_reads_match_line_sets(M, N, K, elt, bm, bn, bk):
    for keep in (False, True):
        pred = tm.predict_l2_reads(M, N, K, elt, bm, bn, bk, l1_keep=1 << 40 if keep else 0)
        assert pred == _l2_brute(M, N, K, elt, bm, bn, bk, keep)


def test_l2_reads_closed_forms():
    M = N = K = 4096
    # whole-line stages (128-byte A runs): each tile reads its panels once
    assert tm.predict_l2_reads(M, N, K, 4, 256, 256, 32) == (M * K * 16 + K * N * 16) * 4
    # half-line A runs (block_k 16) and a stage too large for the L1: every A line twice
    assert tm.predict_l2_reads(M, N, K, 4, 256, 128, 16) == (2 * M * K * 32 + K * N * 16) * 4
    # the same tile alone on its CU with a stage that fits: A lines once
    assert tm.predict_l2_reads(128, 128, K, 4, 128, 128, 16) == (128 * K + K * 128) * 4
    # 1024 tiles: with two resident workgroups per CU the footprint passes the limit
    two = tm.predict_l2_reads(M, N, K, 4, 128, 128, 16, occupancy=2)
    assert two == tm.predict_l2_reads(M, N, K, 4, 128, 128, 16, l1_keep=0) == (2 * M * K * 32 + K * N * 32) * 4
    assert tm.predict_l2_reads(M, N, K, 4, 128, 128, 16, occupancy=1) == (M * K * 32 + K * N * 32) * 4
    # a launch of 16 tiles leaves one workgroup per CU whatever the occupancy
    assert tm.predict_l2_reads(512, 512, K, 4, 128, 128, 16, occupancy=2) == (512 * K * 4 + K * 512 * 4) * 4
    assert tm.predict_l2_reads(0, N, K, 4, 64, 64, 32) == 0


def test_l2_tile_follows_the_fallback():
    s = _sched(block_m=256, block_n=256, block_k=32, lds_pad=-1)
    assert tm.gemm_tile("f32", s, 256, 258, 512) == (128, 128, 32)    # N = 258: rows not whole chunks
    assert tm.gemm_tile("f32", s, 4096, 4096, 4096) == (256, 256, 32)
    assert tm.gemm_tile("bf16", s, 1000, 1000, 1000) == (256, 256, 32)


# TCC_READ_SECTORS_sum x 32 bytes per launch (mean of two), one counter
# pass per shape (a plain 256 MiB copy reads 1.0008 x its bytes):
# (dtype, M, N, K, block_m, block_n, block_k, lds_pad, occupancy) -> bytes
MEASURED_L2 = [
    ("f32", 4096, 4096, 4096, 256, 256, 32, -1, 1, 2150091776),   # whole-line stages
    ("f32", 4096, 4096, 4096, 256, 128, 16, -1, 1, 5361601024),   # A lines twice
    ("f32", 1000, 1000, 1000, 64, 64, 32, -1, 5, 157319104),      # 4000-byte rows, lines kept
    ("f32", 256, 258, 512, 256, 256, 32, -1, 1, 3096192),         # the 128x128 fallback
    ("f32", 32768, 16, 4096, 256, 256, 32, -1, 1, 571819328),     # one 16-column panel
    ("bf16", 2048, 2048, 2048, 256, 256, 32, -1, 1, 201325120),   # bf16 half-line A runs
]


@pytest.mark.parametrize("dtype,M,N,K,bm,bn,bk,pad,occ,measured", MEASURED_L2)
def test_l2_model_against_counters(dtype, M, N, K, bm, bn, bk, pad, occ, measured):
    s = _sched(block_m=bm, block_n=bn, block_k=bk, lds_pad=pad)
    tile = tm.gemm_tile(dtype, s, M, N, K)
    pred = tm.predict_l2_reads(M, N, K, 4 if dtype == "f32" else 2, *tile, occupancy=occ)
    assert 0.95 <= pred / measured <= 1.02


def test_few_channel_conv_grid_and_counters():
    # the patch-staged few-channel kernel: 64-pixel tiles, each reading its
    # 9 patch rows (7x7 stride 2) of every channel; FETCH_SIZE x 1024 x
    # 1.9998 measured 943650 bytes per launch on the paper's 7x7 layer
    s = _sched(block_m=16, block_n=64, block_k=128, wave_m=16, wave_n=16, mfma_m=16, lds_stages=0, lds_pad=0)
    dims = (1, 3, 224, 224, 16, 7, 7, 2, 3)
    bm, tmm, tn, seg, force = tm.conv_grid("f32", s, *dims)
    assert (bm, tmm, tn) == (16, 1, 112 * 112 // 64)
    assert seg(1) == [(0, 0, 5)]        # pixels 64..127: output rows 0..1, patch rows -3..5
    assert seg(2) == [(0, 0, 7)]        # pixels 128..191 start on output row 1: patch rows -1..7
    assert seg(195) == [(0, 219, 223)]  # the last tile: patch rows 219..227, the image ends at 223
    r, w = tm.predict_conv("f32", s, dims, 1)
    assert w == 4 * 16 * 112 * 112 and 0.85 <= r / 943650 <= 0.95
    # the gather form (the patch does not fit) is not modelled
    assert tm.conv_grid("f32", s, 32, 64, 56, 56, 64, 3, 3, 1, 1) is None


def test_conv_l2_reads_row_loads_and_weights():
    # bf16 row-streaming kernel, 32x64x56x56 -> 64: 224 workgroups, each
    # reading its band's 10 input rows (8 for the first and last bands, which
    # start or end in the padding) of 64 channels, each 112-byte row as whole
    # lines of its own, and 64 x 576 weights (72 KiB, 576 lines)
    s = _sched(block_n=64, block_m=64, block_k=16, k_order=3)
    dims = (32, 64, 56, 56, 64, 3, 3, 1, 1)
    got = tm.predict_conv_l2("bf16", s, dims)
    rows = 0
    for img in range(32):
        for band in range(7):
            lo, hi = max(0, band * 8 - 1), min(55, band * 8 + 8)
            for c in range(64):
                for r in range(lo, hi + 1):
                    st = ((img * 64 + c) * 56 + r) * 112
                    rows += (st + 111) // 128 - st // 128 + 1
    assert got == (rows + 224 * 576) * 128
    # measured TCC_READ_SECTORS x 32: 39.65e6 bytes (raster 0, XCD remap)
    assert 1.1 <= got / 39.65e6 <= 1.2
    # the gather kernels are not modelled
    assert tm.predict_conv_l2("f32", _sched(block_n=128, k_order=0, lds_stages=3), dims) is None
