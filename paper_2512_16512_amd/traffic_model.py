"""Analytic model of the HBM traffic of a matmul or conv schedule, and its
evaluation against hardware counters.

The GPU counterpart of the paper's cache-model study (Sec. 6.3, Fig. 13,
Table 2): a model predicts, for every schedule of a design space, the misses
of one cache level; the schedules are run under the counter profiler and the
prediction is compared with the counter by Pearson's r and Spearman's rho.
The paper models the L1 of a CPU core as one fully associative cache; here the
level that decides HBM traffic is the L2 of each of the MI355X's 8 XCDs
(4 MiB each, private), which the L2 miss counters (FETCH_SIZE) measure.

Model.  The dispatcher hands workgroup ids to the XCDs round-robin (id % 8)
and each XCD runs its ids in order, ``occupancy`` workgroups per CU on its 32
CUs at once, so each XCD works through consecutive groups of
``32 * occupancy`` of its tiles (the workgroup -> tile map is the library's
raster order and XCD remap).  Workgroups of one group advance through K at
about the same pace, so an A row-panel or B column-panel shared by several of
them is fetched from HBM once per group; nothing is assumed to survive from
one group to the next, unless everything the XCD touches fits in its L2,
in which case every panel is fetched once per XCD.  Predicted read bytes are
the sum over XCDs and groups of (distinct A row-panels) x rows x K x elt +
(distinct B column-panels) x columns x K x elt; the output is written once
(M x N x 4 bytes).  The model ignores cache-line granularity, the replacement
policy, and timing skew between workgroups.

The last-level cache.  Behind the L2s, the 256 MiB MALL is shared by all
XCDs: an L2 miss that hits there costs no DRAM traffic.  ``predict_dram``
replays the same tile groups, XCDs in lockstep rounds, through a 256 MiB
least-recently-used panel cache and counts the DRAM reads.  No counter
separates MALL hits from DRAM reads (the L2 counters see both as misses),
so that term is evaluated against kernel time over the tile orders
(``orders`` / ``evaluate-orders``), together with the L2 term and their
unweighted sum.

Convolutions (``conv_grid``, ``predict_conv``) follow the same L2 rule with
the launchers' own tile grids; a workgroup's footprint is the weights of its
output-channel tile and the input rows its output rows reach.

The level above.  ``predict_l2_reads`` models what the workgroups of a
matmul read from L2 (TCC_READ_SECTORS): each tile's operand panels, one
K-stage at a time, in whole cache lines, with lines that consecutive stages
share kept only when the resident workgroups' stage blocks fit in half the
CU's L1 (``correlate-l2``).  ``predict_conv_l2`` does the same for the conv
kernels that stage whole input rows (``correlate-conv-l2``).

Usage (the measurement step runs under rocprofv3; see ``run``)::

    rocprofv3 --pmc FETCH_SIZE -f csv -d OUT -o run -- \\
        python3 -m paper_2512_16512_amd.traffic_model run f32 4096 4096 4096 --order ORDER.json
    python -m paper_2512_16512_amd.traffic_model correlate ORDER.json OUT/run_counter_collection.csv \\
        --fetch-scale 2.0
    rocprofv3 --pmc FETCH_SIZE -f csv -d OUT -o run -- \\
        python3 -m paper_2512_16512_amd.traffic_model run-conv f32 32 64 56 56 64 3 3 1 1 --order ORDER.json
    python -m paper_2512_16512_amd.traffic_model correlate-conv ORDER.json OUT/run_counter_collection.csv \\
        --fetch-scale 2.0
    rocprofv3 --pmc TCC_READ_SECTORS_sum -f csv -d OUT -o run -- \\
        python3 -m paper_2512_16512_amd.traffic_model run f32 1000 1000 1000 --order ORDER.json --rasters 0,1
    python -m paper_2512_16512_amd.traffic_model correlate-l2 ORDER.json OUT/run_counter_collection.csv
    rocprofv3 --pmc TCC_READ_SECTORS_sum -f csv -d OUT -o run -- \\
        python3 -m paper_2512_16512_amd.traffic_model run-conv bf16 32 64 56 56 64 3 3 1 1 --order ORDER.json
    python -m paper_2512_16512_amd.traffic_model correlate-conv-l2 ORDER.json OUT/run_counter_collection.csv
"""
from __future__ import annotations

import argparse
import json
import sys

XCDS = 8
CUS_PER_XCD = 32
L2_BYTES = 4 << 20


def tile_coords(bid: int, grid: int, tiles_m: int, tiles_n: int, raster: int, xcd_remap: int):
    """Tile (tm, tn) of workgroup ``bid``: the same map the kernels apply
    (XCD remap into contiguous bands per XCD, then the raster order)."""
    if xcd_remap and grid >= XCDS:
        x, q, rem = bid % XCDS, grid // XCDS, grid % XCDS
        bid = x * q + min(x, rem) + bid // XCDS
    if raster == 1:
        return bid % tiles_m, bid // tiles_m
    if raster >= 2:
        per = raster * tiles_n
        grp = bid // per
        first = grp * raster
        gsz = min(tiles_m - first, raster)
        r = bid - grp * per
        return first + r % gsz, r // gsz
    return bid // tiles_n, bid % tiles_n


def predict(M: int, N: int, K: int, elt: int, block_m: int, block_n: int, raster: int,
            xcd_remap: int, occupancy: int, l2_bytes: int = L2_BYTES):
    """Predicted HBM (read, write) bytes of one launch."""
    tiles_m = -(-M // block_m)
    tiles_n = -(-N // block_n)
    grid = tiles_m * tiles_n
    rows = [min(block_m, M - t * block_m) for t in range(tiles_m)]
    cols = [min(block_n, N - t * block_n) for t in range(tiles_n)]
    conc = max(1, CUS_PER_XCD * max(1, occupancy))
    read = 0
    for x in range(XCDS):
        ids = range(x, grid, XCDS)
        tiles = [tile_coords(b, grid, tiles_m, tiles_n, raster, xcd_remap) for b in ids]
        all_m = {t[0] for t in tiles}
        all_n = {t[1] for t in tiles}
        footprint = (sum(rows[m] for m in all_m) + sum(cols[n] for n in all_n)) * K * elt
        if footprint <= l2_bytes:
            read += footprint
            continue
        for g0 in range(0, len(tiles), conc):
            grp = tiles[g0:g0 + conc]
            read += (sum(rows[m] for m in {t[0] for t in grp}) +
                     sum(cols[n] for n in {t[1] for t in grp})) * K * elt
    return read, 4 * M * N


MALL_BYTES = 256 << 20


def predict_dram(M: int, N: int, K: int, elt: int, block_m: int, block_n: int, raster: int,
                 xcd_remap: int, occupancy: int, mall_bytes: int = MALL_BYTES):
    """Predicted DRAM read bytes of one launch, with the last-level cache
    (MALL, 256 MiB on MI355X, shared by the 8 XCDs) in front of HBM.

    The XCDs advance through their groups of ``32 * occupancy`` tiles in
    lockstep rounds (the same groups as ``predict``).  In a round every XCD
    asks the MALL for the A row-panels and B column-panels of its group; a
    panel the MALL holds is a hit, any other is read from DRAM once for all
    the XCDs that ask for it in that round and then kept, least recently used
    first out, within ``mall_bytes``.  The L2 misses ``predict`` counts are
    the MALL requests; the difference is what the XCDs share in the MALL."""
    from collections import OrderedDict
    tiles_m = -(-M // block_m)
    tiles_n = -(-N // block_n)
    grid = tiles_m * tiles_n
    conc = max(1, CUS_PER_XCD * max(1, occupancy))
    groups = []
    for x in range(XCDS):
        ids = list(range(x, grid, XCDS))
        tiles = [tile_coords(b, grid, tiles_m, tiles_n, raster, xcd_remap) for b in ids]
        groups.append([tiles[g0:g0 + conc] for g0 in range(0, len(tiles), conc)])
    rounds = max(len(g) for g in groups)
    panel_bytes = lambda p: (min(block_m, M - p[1] * block_m) if p[0] == "A"
                             else min(block_n, N - p[1] * block_n)) * K * elt
    mall = OrderedDict()
    held = 0
    dram = 0
    for r in range(rounds):
        want = []
        for g in groups:
            if r < len(g):
                want += [("A", t[0]) for t in g[r]] + [("B", t[1]) for t in g[r]]
        for p in dict.fromkeys(want):
            if p in mall:
                mall.move_to_end(p)
                continue
            nb = panel_bytes(p)
            dram += nb
            mall[p] = nb
            held += nb
            while held > mall_bytes and len(mall) > 1:
                _, old = mall.popitem(last=False)
                held -= old
    return dram


def _ranks(v):
    """Ranks 1..n with ties given their average rank."""
    order = sorted(range(len(v)), key=lambda i: v[i])
    r = [0.0] * len(v)
    i = 0
    while i < len(order):
        j = i
        while j + 1 < len(order) and v[order[j + 1]] == v[order[i]]:
            j += 1
        avg = (i + j) / 2.0 + 1.0
        for k in range(i, j + 1):
            r[order[k]] = avg
        i = j + 1
    return r


def pearson(x, y) -> float:
    n = len(x)
    mx, my = sum(x) / n, sum(y) / n
    sxy = sum((a - mx) * (b - my) for a, b in zip(x, y))
    sxx = sum((a - mx) ** 2 for a in x)
    syy = sum((b - my) ** 2 for b in y)
    if sxx == 0 or syy == 0:
        return float("nan")   # undefined for a constant series
    return sxy / (sxx * syy) ** 0.5


def spearman(x, y) -> float:
    return pearson(_ranks(x), _ranks(y))


# ---------------------------------------------------------------- measuring


def run(dtype: str, M: int, N: int, K: int, order_path: str, reps: int = 2, rasters=(0, 1, 4, 8, 16)):
    """Launch every schedule of the design space ``reps`` times, in a fixed
    order, and write that order (with each schedule's occupancy) to
    ``order_path``, so that the profiler's per-dispatch counter rows can be
    matched to schedules afterwards."""
    import torch

    import paper_2512_16512_amd as xtc
    from paper_2512_16512_amd import tune
    p = tune.Problem("matmul", dtype, (M, N, K))
    space = tune.design_space(xtc.XTC_OP_MATMUL, p.code, rasters=rasters)
    entries = []
    stream = torch.cuda.current_stream().cuda_stream
    for s in space:
        occ = xtc.xtc_sched_occupancy(xtc.XTC_OP_MATMUL, p.code, K, s)
        for _ in range(reps):
            p.launch(s, stream)
        torch.cuda.synchronize()
        entries.append({"sched": s.as_dict(), "occupancy": occ})
    with open(order_path, "w") as f:
        json.dump({"dtype": dtype, "M": M, "N": N, "K": K, "reps": reps, "schedules": entries}, f)
    print("launched %d schedules x %d" % (len(entries), reps), flush=True)


ORDERS = tuple((r, x) for r in (0, 1, 2, 4, 8, 16, 32) for x in (0, 1))


def sweep_orders(dtype: str, M: int, N: int, K: int, out_path: str, warmup: int = 2, reps: int = 5,
                 passes: int = 3, warm_s: float = 0.5):
    """Time the default schedule of one matmul under every tile order
    (raster x XCD remap in ORDERS).  After ``warm_s`` seconds of untimed
    launches (the clock settles), ``passes`` passes over the orders each run
    ``warmup`` untimed launches and ``reps`` launches between their own HIP
    events per order; an order's time is the median of its ``passes * reps``
    launches.  Writes the times, the launch order (``warmup + reps``
    dispatches per order and pass, after the warm-up dispatches, for
    matching a counter pass) and the schedule's occupancy to ``out_path``."""
    import torch

    import paper_2512_16512_amd as xtc
    from paper_2512_16512_amd import tune
    p = tune.Problem("matmul", dtype, (M, N, K))
    base = xtc.xtc_default_schedule(xtc.XTC_OP_MATMUL, p.code, M, N, K)
    occ = xtc.xtc_sched_occupancy(xtc.XTC_OP_MATMUL, p.code, K, base)
    stream = torch.cuda.current_stream().cuda_stream
    import time
    nwarm = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < warm_s:
        for _ in range(4):
            p.launch(base, stream)
        nwarm += 4
        torch.cuda.synchronize()
    times = {o: [] for o in ORDERS}
    for _ in range(passes):
        for raster, remap in ORDERS:
            s = xtc.Sched(**base.as_dict())
            s.raster, s.xcd_remap = raster, remap
            for _ in range(warmup):
                p.launch(s, stream)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(reps)]
            for e0, e1 in ev:
                e0.record()
                p.launch(s, stream)
                e1.record()
            torch.cuda.synchronize()
            times[(raster, remap)] += [e0.elapsed_time(e1) for e0, e1 in ev]
    rows = []
    for raster, remap in ORDERS:
        t = sorted(times[(raster, remap)])
        rows.append({"raster": raster, "xcd_remap": remap, "median_ms": t[len(t) // 2]})
    with open(out_path, "w") as f:
        json.dump({"dtype": dtype, "M": M, "N": N, "K": K, "warmup": warmup, "reps": reps,
                   "passes": passes, "warm_dispatches": nwarm, "sched": base.as_dict(),
                   "occupancy": occ, "orders": rows}, f)
    print("timed %d tile orders" % len(rows), flush=True)


def evaluate_orders(sweep_path: str, fetch_csv: str = None, fetch_scale: float = 2.0,
                    fetch_order: str = None):
    """Per tile order: the L2-miss bytes ``predict`` gives, the DRAM bytes
    ``predict_dram`` gives, the measured time and (with a FETCH_SIZE pass
    of the same sweep) the measured L2-miss bytes; returns the rows and the
    Pearson / Spearman coefficients of each prediction against time (and of
    the L2-miss prediction against FETCH_SIZE).  ``fetch_order`` is the
    record the counter pass wrote (its warm-up count may differ from the
    timing pass's); the timing pass's own record by default."""
    o = json.load(open(sweep_path))
    fo = json.load(open(fetch_order)) if fetch_order else o
    s = o["sched"]
    elt = 4 if o["dtype"] == "f32" else 2
    fetch = None
    if fetch_csv:
        vals = _counter_rows(fetch_csv, "FETCH_SIZE")
        per, nord, npass = fo["warmup"] + fo["reps"], len(fo["orders"]), fo.get("passes", 1)
        skip = fo.get("warm_dispatches", 0)
        if len(vals) != skip + npass * per * nord:
            raise ValueError("%d counter rows for %d + %d passes x %d orders x %d launches"
                             % (len(vals), skip, npass, nord, per))
        fetch = []
        for i in range(nord):
            got = [v for q in range(npass)
                   for v in vals[skip + (q * nord + i) * per + fo["warmup"]:skip + (q * nord + i + 1) * per]]
            fetch.append(sum(got) / len(got) * 1024 * fetch_scale)
    rows = []
    for i, r in enumerate(o["orders"]):
        l2, _ = predict(o["M"], o["N"], o["K"], elt, s["block_m"], s["block_n"], r["raster"],
                        r["xcd_remap"], o["occupancy"])
        dram = predict_dram(o["M"], o["N"], o["K"], elt, s["block_m"], s["block_n"], r["raster"],
                            r["xcd_remap"], o["occupancy"])
        rows.append(dict(r, l2_pred=l2, dram_pred=dram, fetch=None if fetch is None else fetch[i]))
    t = [r["median_ms"] for r in rows]
    comb = [r["l2_pred"] + r["dram_pred"] for r in rows]
    stats = {"l2_vs_time": (pearson([r["l2_pred"] for r in rows], t), spearman([r["l2_pred"] for r in rows], t)),
             "dram_vs_time": (pearson([r["dram_pred"] for r in rows], t),
                              spearman([r["dram_pred"] for r in rows], t)),
             "l2+dram_vs_time": (pearson(comb, t), spearman(comb, t))}
    if fetch is not None:
        stats["l2_vs_fetch"] = (pearson([r["l2_pred"] for r in rows], fetch),
                                spearman([r["l2_pred"] for r in rows], fetch))
    return rows, stats


def _counter_rows(csv_path: str, counter: str):
    import csv
    rows = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] != counter or "xtc::" not in r["Kernel_Name"]:
            continue
        d = int(r["Dispatch_Id"])
        rows[d] = rows.get(d, 0.0) + float(r["Counter_Value"])
    return [rows[d] for d in sorted(rows)]


def correlate(order_path: str, fetch_csv: str, fetch_scale: float):
    """Predicted vs measured (FETCH_SIZE x 1024 x fetch_scale) bytes per
    schedule; returns the table rows and the two correlation statistics."""
    o = json.load(open(order_path))
    vals = _counter_rows(fetch_csv, "FETCH_SIZE")
    reps = o["reps"]
    if len(vals) != reps * len(o["schedules"]):
        raise ValueError("%d counter rows for %d schedules x %d launches"
                         % (len(vals), len(o["schedules"]), reps))
    elt = 4 if o["dtype"] == "f32" else 2
    table = []
    for i, e in enumerate(o["schedules"]):
        s = e["sched"]
        meas = sum(vals[i * reps:(i + 1) * reps]) / reps * 1024 * fetch_scale
        pred, _ = predict(o["M"], o["N"], o["K"], elt, s["block_m"], s["block_n"], s["raster"],
                          s["xcd_remap"], e["occupancy"])
        table.append({"sched": s, "occupancy": e["occupancy"], "predicted": pred,
                      "measured": meas})
    x = [t["predicted"] for t in table]
    y = [t["measured"] for t in table]
    return table, pearson(x, y), spearman(x, y)


# ------------------------------------------------ L2 reads (the CU side)

SECTOR = 32            # bytes per L2 read sector (the unit of TCC_READ_SECTORS)
LINE = 128             # bytes per cache line
L1_KEEP = 16 << 10     # half the CU's 32 KiB vector L1 (see ``predict_l2_reads``)


def _block_lines(starts, length: int, line: int = LINE) -> int:
    """Distinct lines of ``line`` bytes touched by byte runs of ``length``
    at the increasing, non-overlapping offsets ``starts`` (a run can share
    a line only with its neighbours)."""
    import numpy as np
    st = np.asarray(starts, dtype=np.int64)
    if length <= 0 or st.size == 0:
        return 0
    first, last = st // line, (st + length - 1) // line
    return int((last - first + 1).sum() - (last[:-1] >= first[1:]).sum())


def gemm_tile(dtype: str, s: dict, M: int, N: int, K: int):
    """(block_m, block_n, block_k) of the kernel a matmul instance runs on
    this shape (contiguous operands, 16-byte aligned bases): the fp32
    256x256 direct-to-LDS instances fall back to the register-staged
    128x128x32 kernel when K or N is not a whole number of 16-byte chunks;
    every other instance keeps its tile."""
    elt = 4 if dtype == "f32" else 2
    whole = (K * elt) % 16 == 0 and (N * elt) % 16 == 0
    if dtype == "f32" and s["lds_pad"] == -1 and s["block_m"] == 256 and s["block_n"] == 256 and not whole:
        return 128, 128, 32
    return s["block_m"], s["block_n"], s["block_k"]


def predict_l2_reads(M: int, N: int, K: int, elt: int, block_m: int, block_n: int, block_k: int,
                     occupancy: int = 1, lda: int = None, ldb: int = None, l1_keep: int = L1_KEEP,
                     line: int = LINE) -> int:
    """Bytes the workgroups of one matmul launch read from L2, for the
    kernels that stage their operands through LDS (the level above the one
    ``predict`` models).

    Every output tile reads the in-range part of its A row-panel and B
    column-panel one K-stage at a time: per stage an A block (rows x
    block_k) and a B block (block_k rows x columns), each fetched as the
    distinct cache lines its rows touch.  A line that two consecutive
    stages share (a stage's A rows are half a line for fp32 with block_k 16
    or bf16 with block_k 32; rows not aligned to a line) is fetched again
    unless it survives in the CU's L1 from one stage to the next, which the
    model takes to happen when the stage blocks of the workgroups resident
    on a CU (min(occupancy, tiles per CU)) fit in half the L1; the panel's
    distinct lines are then fetched once.  Reuse between workgroups is not
    modelled.  Out-of-range elements (ragged edges) are not read."""
    import numpy as np
    if M <= 0 or N <= 0 or K <= 0:
        return 0
    lda = K if lda is None else lda
    ldb = N if ldb is None else ldb
    tiles_m, tiles_n = _cdiv(M, block_m), _cdiv(N, block_n)
    resident = min(max(1, occupancy), _cdiv(tiles_m * tiles_n, XCDS * CUS_PER_XCD))
    keep = resident * (min(block_m, M) + min(block_n, N)) * block_k * elt <= l1_keep
    stages = [(k0, min(block_k, K - k0)) for k0 in range(0, K, block_k)]
    a = b = 0
    for t in range(tiles_m):
        rows = np.arange(t * block_m, min(M, (t + 1) * block_m), dtype=np.int64) * lda * elt
        if keep:
            a += _block_lines(rows, K * elt, line)
        else:
            a += sum(_block_lines(rows + k0 * elt, kk * elt, line) for k0, kk in stages)
    for t in range(tiles_n):
        n0, cols = t * block_n, min(block_n, N - t * block_n)
        if keep:
            b += _block_lines(np.arange(K, dtype=np.int64) * ldb * elt + n0 * elt, cols * elt, line)
        else:
            b += sum(_block_lines(np.arange(k0, k0 + kk, dtype=np.int64) * ldb * elt + n0 * elt,
                                  cols * elt, line) for k0, kk in stages)
    return (a * tiles_n + b * tiles_m) * line


def correlate_l2(order_path: str, csv_path: str):
    """Predicted (``predict_l2_reads``) vs measured (TCC_READ_SECTORS x 32)
    L2 read bytes per matmul schedule of a ``run`` order file.  The
    register-fed reduction-split kernels (no LDS stages), which read their
    MFMA fragments straight from memory, are not modelled (predicted None);
    the statistics are over the modelled schedules."""
    o = json.load(open(order_path))
    vals = _counter_rows(csv_path, "TCC_READ_SECTORS_sum")
    reps = o["reps"]
    if len(vals) != reps * len(o["schedules"]):
        raise ValueError("%d counter rows for %d schedules x %d launches"
                         % (len(vals), len(o["schedules"]), reps))
    M, N, K = o["M"], o["N"], o["K"]
    elt = 4 if o["dtype"] == "f32" else 2
    table = []
    for i, e in enumerate(o["schedules"]):
        s = e["sched"]
        meas = sum(vals[i * reps:(i + 1) * reps]) / reps * SECTOR
        pred = None
        if s["lds_stages"] > 0:
            bm, bn, bk = gemm_tile(o["dtype"], s, M, N, K)
            pred = predict_l2_reads(M, N, K, elt, bm, bn, bk, e["occupancy"])
        table.append({"sched": s, "occupancy": e["occupancy"], "predicted": pred, "measured": meas})
    mod = [t for t in table if t["predicted"] is not None]
    x = [t["predicted"] for t in mod]
    y = [t["measured"] for t in mod]
    return table, pearson(x, y), spearman(x, y)


# ------------------------------------------------------------------- conv

def _cdiv(a: int, b: int) -> int:
    return -(-a // b)


def conv_grid(dtype: str, s: dict, N, C, H, W, OC, R, S, stride, pad):
    """The tile grid of the kernel the library runs for conv instance ``s``
    on this shape: (BM, tiles_m, tiles_n, segments, forced XCD remap or
    None), where ``segments(tn)`` lists the (image, first output row, last
    output row, input rows read) of pixel tile ``tn``.  Follows the
    launchers' choice of kernel and tile (the balanced halo kernel's pixel
    tile, the row-streaming kernel's bands, the fallbacks outside a kernel's
    class); None where the choice is not modelled."""
    sh = sw = stride
    ph = pw = pad
    OH, OW = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    OHW = OH * OW
    halo_class = R == 3 and S == 3 and sh == 1 and sw == 1

    def rows_of(oh0, oh1):
        return max(0, oh0 * sh - ph), min(H - 1, oh1 * sh - ph + R - 1)

    def per_image(pt):
        chunks = _cdiv(OHW, pt)

        def seg(tn):
            img, c = divmod(tn, chunks)
            p0, p1 = c * pt, min((c + 1) * pt, OHW)
            oh0, oh1 = p0 // OW, (p1 - 1) // OW
            return [(img,) + rows_of(oh0, oh1)]
        return N * chunks, seg

    def flattened(bn):
        tot = N * OHW

        def seg(tn):
            q0, q1 = tn * bn, min((tn + 1) * bn, tot)
            out = []
            while q0 < q1:
                img, p0 = divmod(q0, OHW)
                p1 = min(q1 - img * OHW, OHW)
                out.append((img,) + rows_of(p0 // OW, (p1 - 1) // OW))
                q0 = img * OHW + p1
            return out
        return _cdiv(tot, bn), seg

    bm, force = s["block_m"], None
    if dtype == "bf16" and s["k_order"] == 3:
        if halo_class and C == 64 and W % 2 == 0 and pw <= 2 and OW % 4 == 0 and OW <= 64 and OW + 1 - pw + 2 <= 63:
            per_img = _cdiv(OC, 64) * N
            band = _cdiv(_cdiv(OH, _cdiv(256, per_img)), 2) * 2    # whole 2-row steps
            nb = _cdiv(OH, band)

            def seg(tn):
                img, b = divmod(tn, nb)
                rows = min(band, OH - b * band)
                nin = 2 * _cdiv(rows, 2) + 2          # the band's input rows, as the kernel reads them
                lo = b * band - ph
                return [(img, max(0, lo), min(H - 1, lo + nin - 1))]
            return 64, _cdiv(OC, 64), N * nb, seg, 1
        s = dict(s, k_order=2, block_n=256)
    if dtype == "bf16" and s["k_order"] == 2:
        span = (256 - 1 + OW - 1) // OW + 1
        if halo_class and C % 16 == 0 and W % 2 == 0 and pw <= 2 and OW - pw + 3 <= 63 and span + 2 <= 8:
            tn, seg = per_image(256)
            return 64, _cdiv(OC, 64), tn, seg, None
        s = dict(s, block_m=64, block_n=128)           # the gather kernel's 64x128 tiles
        bm = 64
    if dtype == "bf16":
        tn, seg = flattened(s["block_n"])
        return bm, _cdiv(OC, bm), tn, seg, None
    if s["k_order"] == 2 and s["block_n"] in (208, 416):
        nh = 1 if s["block_n"] == 208 else 2
        if halo_class and C % 8 == 0 and pw <= 4 and OW - pw + 5 <= 63:
            t = _cdiv(OHW, 208 * nh)
            pt = _cdiv(OHW, t)
            if (pt - 1 + OW - 1) // OW + 1 + 2 <= (8 if nh == 1 else 10):
                tn, seg = per_image(pt)
                return 64, _cdiv(OC, 64), tn, seg, None
        s = dict(s, block_n=256)
    if s["k_order"] == 2:
        span = (256 - 1 + OW - 1) // OW + 1
        if halo_class and C % 16 == 0 and pw <= 4 and OW - pw + 5 <= 63 and span + 2 <= 8:
            tn, seg = per_image(256)
            return 64, _cdiv(OC, 64), tn, seg, None
        tn, seg = flattened(256)                       # the tap-major 64x256 fallback
        return 64, _cdiv(OC, 64), tn, seg, None
    if bm == 16:
        # few output channels: 64-pixel tiles; the patch-staged form loads, per
        # tile, its patch rows of every channel (rows outside the image read
        # nothing); the gather form (the patch does not fit) is not modelled
        bn = 64
        span = (bn - 1 + OW - 1) // OW + 1
        PR = (span - 1) * sh + R
        vec = W % 4 == 0
        padl = (pw + 3) // 4 * 4 if vec else pw
        WP = (OW - 1) * sw + S - pw + padl
        if vec:
            WP = (WP + 3) // 4 * 4
        K = C * R * S
        kp = _cdiv(K, 32) * 32
        area = max(C * PR * WP, 32 * bn)
        if not (4 * (area + 16 * (kp + 2)) + 4 * kp <= 48 * 1024 and WP <= 256 and kp <= 256):
            return None
        chunks = _cdiv(OHW, bn)

        def seg(tn):
            img, c = divmod(tn, chunks)
            lo = (c * bn // OW) * sh - ph
            return [(img, max(0, lo), min(H - 1, lo + PR - 1))]
        return 16, _cdiv(OC, 16), N * chunks, seg, None
    tn, seg = flattened(s["block_n"])
    return bm, _cdiv(OC, bm), tn, seg, None


def predict_conv(dtype: str, s: dict, dims, occupancy: int, l2_bytes: int = L2_BYTES):
    """Predicted HBM (read, write) bytes of one conv launch of instance
    ``s`` (``dims`` = N, C, H, W, OC, R, S, stride, pad), or None where the
    kernel's tiles are not modelled.

    A workgroup reads the weights of its output-channel tile and, of each
    image its pixel tile touches, every input row its output rows reach
    (all channels, whole rows).  As in ``predict``, an XCD whose workgroups
    together touch at most its L2 reads each row and weight panel once;
    otherwise each group of ``32 * occupancy`` workgroups that run at once
    reads the union of what it touches.  The output is written once."""
    N, C, H, W, OC, R, S, stride, pad = dims
    g = conv_grid(dtype, s, *dims)
    if g is None:
        return None
    bm, tiles_m, tiles_n, seg, force = g
    raster = s["raster"]
    remap = s["xcd_remap"] if force is None else force
    elt = 4 if dtype == "f32" else 2
    row_bytes = C * W * elt
    K = C * R * S
    grid = tiles_m * tiles_n
    conc = max(1, CUS_PER_XCD * max(1, occupancy))

    def footprint(tiles):
        wts = {t[0] for t in tiles}
        rows = set()
        for t in tiles:
            for img, lo, hi in seg(t[1]):
                rows.update((img, r) for r in range(lo, hi + 1))
        return sum(min(bm, OC - m * bm) for m in wts) * K * elt + len(rows) * row_bytes

    read = 0
    for x in range(XCDS):
        tiles = [tile_coords(b, grid, tiles_m, tiles_n, raster, remap) for b in range(x, grid, XCDS)]
        if not tiles:
            continue
        f = footprint(tiles)
        if f <= l2_bytes:
            read += f
            continue
        read += sum(footprint(tiles[g0:g0 + conc]) for g0 in range(0, len(tiles), conc))
    OH, OW = (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1
    return read, 4 * N * OC * OH * OW


def predict_conv_l2(dtype: str, s: dict, dims, line: int = LINE):
    """Bytes the workgroups of one conv launch read from L2, for the kernels
    that stage whole input rows (None for the others, whose gathers re-read
    inputs through the L1 tap by tap): every workgroup reads, per channel
    it stages, its patch or band rows inside the image as one contiguous
    run, and its weights, each run in whole cache lines, with no reuse
    between stages or workgroups.
      - fp32 halo kernel (k_order 2, 64x208 or 64x416 tiles): per 8-channel
        stage, 8 (one pixel half) or 10 (two) patch rows from the tile's
        first output row less the padding, and the stage's 64 x 8 x 9
        weights (one 288-byte run per output channel);
      - bf16 row-streaming kernel (k_order 3): the band's input rows of all
        64 channels and the 64 output channels' 576 weights each;
      - few-channel kernel (block_m 16, patch-staged): its patch rows of
        every channel and its 16 output channels' weights."""
    import numpy as np
    N, C, H, W, OC, R, S, stride, pad = dims
    g = conv_grid(dtype, s, *dims)
    if g is None:
        return None
    bm, tiles_m, tiles_n, seg, force = g
    elt = 4 if dtype == "f32" else 2
    OH, OW = (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1
    K = C * R * S

    def rows_run(img, c, lo, hi):
        # each input row is its own load (its own instructions, at its own
        # time), so a line two neighbouring rows share is fetched for each
        if hi < lo:
            return 0
        starts = (((img * C + c) * H + np.arange(lo, hi + 1, dtype=np.int64)) * W * elt)
        return int(((starts + W * elt - 1) // line - starts // line + 1).sum())

    def weights(m, width):
        rows = np.arange(m * bm, min(OC, (m + 1) * bm), dtype=np.int64)
        return _block_lines(rows * K * elt, width * elt, line) if rows.size else 0

    total = 0
    halo16 = (dtype == "f32" and s["k_order"] == 2 and s["block_n"] in (208, 416) and R == 3 and S == 3
              and stride == 1 and C % 8 == 0 and pad <= 4 and OW - pad + 5 <= 63 and tiles_n % N == 0
              and tiles_n // N == _cdiv(OH * OW, 208 * (1 if s["block_n"] == 208 else 2)))
    if halo16:
        PR = 8 if s["block_n"] == 208 else 10
        ohw = OH * OW
        chunks = tiles_n // N
        pt = _cdiv(ohw, chunks)
        rows_total = 0
        for img in range(N):
            for ch in range(chunks):
                lo = (ch * pt) // OW - pad
                a, b = max(0, lo), min(H - 1, lo + PR - 1)
                rows_total += sum(rows_run(img, c, a, b) for c in range(C))
        for m in range(tiles_m):
            oc = np.arange(m * bm, min(OC, (m + 1) * bm), dtype=np.int64)
            w = sum(_block_lines(oc * K * 4 + c0 * 9 * 4, 8 * 9 * 4, line) for c0 in range(0, C, 8))
            total += rows_total + w * tiles_n
        return total * line
    if (dtype == "bf16" and s["k_order"] == 3 and force == 1) or bm == 16:
        per_tile_rows = 0
        for tn in range(tiles_n):
            for img, lo, hi in seg(tn):
                per_tile_rows += sum(rows_run(img, c, lo, hi) for c in range(C))
        for m in range(tiles_m):
            total += per_tile_rows + weights(m, K) * tiles_n
        return total * line
    return None


CONV_ORDERS = ((0, 1), (0, 0), (1, 1), (1, 0), (8, 1))


def run_conv(dtype: str, dims, order_path: str, reps: int = 2, orders=CONV_ORDERS):
    """Launch every conv instance under every tile order in ``orders``
    ``reps`` times, in a fixed order, and write that order (with each
    schedule's occupancy) to ``order_path`` (the measurement step of
    ``correlate_conv``, run under the counter profiler)."""
    import torch

    import paper_2512_16512_amd as xtc
    from paper_2512_16512_amd import tune
    p = tune.Problem("conv2d", dtype, tuple(dims))
    N, C, H, W, OC, R, S, stride, pad = dims
    entries = []
    stream = torch.cuda.current_stream().cuda_stream
    for base in xtc.xtc_sched_list(xtc.XTC_OP_CONV2D, p.code):
        for raster, remap in orders:
            s = xtc.Sched(**base.as_dict())
            s.raster, s.xcd_remap = raster, remap
            occ = xtc.xtc_sched_occupancy(xtc.XTC_OP_CONV2D, p.code, C * R * S, s)
            for _ in range(reps):
                p.launch(s, stream)
            torch.cuda.synchronize()
            entries.append({"sched": s.as_dict(), "occupancy": occ})
    with open(order_path, "w") as f:
        json.dump({"dtype": dtype, "dims": list(dims), "reps": reps, "schedules": entries}, f)
    print("launched %d conv schedules x %d" % (len(entries), reps), flush=True)


def correlate_conv(order_path: str, fetch_csv: str, fetch_scale: float):
    """Predicted vs measured (FETCH_SIZE x 1024 x fetch_scale) bytes per
    conv schedule; the correlation is over the modelled schedules."""
    o = json.load(open(order_path))
    vals = _counter_rows(fetch_csv, "FETCH_SIZE")
    reps = o["reps"]
    if len(vals) != reps * len(o["schedules"]):
        raise ValueError("%d counter rows for %d schedules x %d launches"
                         % (len(vals), len(o["schedules"]), reps))
    table = []
    for i, e in enumerate(o["schedules"]):
        meas = sum(vals[i * reps:(i + 1) * reps]) / reps * 1024 * fetch_scale
        pred = predict_conv(o["dtype"], e["sched"], tuple(o["dims"]), e["occupancy"])
        table.append({"sched": e["sched"], "occupancy": e["occupancy"],
                      "predicted": None if pred is None else pred[0], "measured": meas})
    mod = [t for t in table if t["predicted"] is not None]
    x = [t["predicted"] for t in mod]
    y = [t["measured"] for t in mod]
    return table, pearson(x, y), spearman(x, y)


def correlate_conv_l2(order_path: str, csv_path: str):
    """Predicted (``predict_conv_l2``) vs measured (TCC_READ_SECTORS x 32)
    L2 read bytes per conv schedule of a ``run-conv`` order file; the
    statistics are over the modelled schedules."""
    o = json.load(open(order_path))
    vals = _counter_rows(csv_path, "TCC_READ_SECTORS_sum")
    reps = o["reps"]
    if len(vals) != reps * len(o["schedules"]):
        raise ValueError("%d counter rows for %d schedules x %d launches"
                         % (len(vals), len(o["schedules"]), reps))
    table = []
    for i, e in enumerate(o["schedules"]):
        meas = sum(vals[i * reps:(i + 1) * reps]) / reps * SECTOR
        pred = predict_conv_l2(o["dtype"], e["sched"], tuple(o["dims"]))
        table.append({"sched": e["sched"], "predicted": pred, "measured": meas})
    mod = [t for t in table if t["predicted"] is not None]
    x = [t["predicted"] for t in mod]
    y = [t["measured"] for t in mod]
    return table, pearson(x, y), spearman(x, y)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    r = sub.add_parser("run")
    r.add_argument("dtype", choices=["f32", "bf16"])
    r.add_argument("M", type=int)
    r.add_argument("N", type=int)
    r.add_argument("K", type=int)
    r.add_argument("--order", required=True)
    r.add_argument("--reps", type=int, default=2)
    r.add_argument("--rasters", default="0,1,4,8,16", help="tile orders, comma-separated")
    w = sub.add_parser("orders")
    w.add_argument("dtype", choices=["f32", "bf16"])
    w.add_argument("M", type=int)
    w.add_argument("N", type=int)
    w.add_argument("K", type=int)
    w.add_argument("--out", required=True)
    e = sub.add_parser("evaluate-orders")
    e.add_argument("sweep")
    e.add_argument("--fetch-csv", default=None)
    e.add_argument("--fetch-scale", type=float, default=2.0)
    e.add_argument("--fetch-order", default=None)
    c = sub.add_parser("correlate")
    c.add_argument("order")
    c.add_argument("fetch_csv")
    c.add_argument("--fetch-scale", type=float, required=True)
    c.add_argument("--json", default=None)
    rc = sub.add_parser("run-conv")
    rc.add_argument("dtype", choices=["f32", "bf16"])
    rc.add_argument("dims", type=int, nargs=9, help="N C H W OC R S stride pad")
    rc.add_argument("--order", required=True)
    rc.add_argument("--reps", type=int, default=2)
    cl = sub.add_parser("correlate-l2")
    cl.add_argument("order")
    cl.add_argument("csv")
    cl.add_argument("--json", default=None)
    cv = sub.add_parser("correlate-conv-l2")
    cv.add_argument("order")
    cv.add_argument("csv")
    cc = sub.add_parser("correlate-conv")
    cc.add_argument("order")
    cc.add_argument("fetch_csv")
    cc.add_argument("--fetch-scale", type=float, required=True)
    cc.add_argument("--json", default=None)
    a = ap.parse_args(argv)
    if a.cmd == "run":
        run(a.dtype, a.M, a.N, a.K, a.order, a.reps, tuple(int(v) for v in a.rasters.split(",")))
        return 0
    if a.cmd == "run-conv":
        run_conv(a.dtype, tuple(a.dims), a.order, a.reps)
        return 0
    if a.cmd == "correlate-l2":
        table, r_, rho = correlate_l2(a.order, a.csv)
        ratio = sorted(t["predicted"] / t["measured"] for t in table if t["predicted"] is not None)
        print("schedules %d (modelled %d)  Pearson r = %.4f  Spearman rho = %.4f  "
              "predicted/measured %.3f .. %.3f" % (len(table), len(ratio), r_, rho, ratio[0], ratio[-1]))
        if a.json:
            with open(a.json, "w") as f:
                json.dump({"pearson": r_, "spearman": rho, "rows": table}, f, indent=1)
        return 0
    if a.cmd == "correlate-conv-l2":
        table, r_, rho = correlate_conv_l2(a.order, a.csv)
        for t in table:
            if t["predicted"] is not None:
                print("%s  predicted %.4g  measured %.4g  %.3f" % (
                    {k: t["sched"][k] for k in ("block_m", "block_n", "k_order", "raster", "xcd_remap")},
                    t["predicted"], t["measured"], t["predicted"] / t["measured"]))
        return 0
    if a.cmd == "correlate-conv":
        table, r_, rho = correlate_conv(a.order, a.fetch_csv, a.fetch_scale)
        n = sum(t["predicted"] is not None for t in table)
        print("conv schedules %d (modelled %d)  Pearson r = %.3f  Spearman rho = %.3f" % (len(table), n, r_, rho))
        if a.json:
            with open(a.json, "w") as f:
                json.dump({"pearson": r_, "spearman": rho, "rows": table}, f, indent=1)
        return 0
    if a.cmd == "orders":
        sweep_orders(a.dtype, a.M, a.N, a.K, a.out)
        return 0
    if a.cmd == "evaluate-orders":
        rows, stats = evaluate_orders(a.sweep, a.fetch_csv, a.fetch_scale, a.fetch_order)
        for r in rows:
            print("raster %2d xcd %d  %.4f ms  L2 pred %.2f GB  DRAM pred %.3f GB%s" % (
                r["raster"], r["xcd_remap"], r["median_ms"], r["l2_pred"] / 1e9, r["dram_pred"] / 1e9,
                "" if r["fetch"] is None else "  FETCH %.2f GB" % (r["fetch"] / 1e9)))
        for k, (r_, rho) in stats.items():
            print("%-14s Pearson r = %.3f  Spearman rho = %.3f" % (k, r_, rho))
        return 0
    table, r_, rho = correlate(a.order, a.fetch_csv, a.fetch_scale)
    print("schedules %d  Pearson r = %.3f  Spearman rho = %.3f" % (len(table), r_, rho))
    if a.json:
        with open(a.json, "w") as f:
            json.dump({"pearson": r_, "spearman": rho, "rows": table}, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
