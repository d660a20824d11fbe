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
