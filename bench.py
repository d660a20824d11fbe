"""Throughput of the tiled dense contraction on one MI355X.

A step is one launch of the contraction on the headline workload: the fp32
matmul M = N = K = 4096 (row-major, uniform [-1, 1) inputs from a fixed seed,
already resident in HBM).  ``value`` is its TFLOP/s (2*M*N*K per launch over
the HIP-event time of exactly ``--steps`` launches, after ``--warmup``
untimed ones, extended to at least 100 ms of launches); ``median_TFLOP/s``
is the per-launch median of further launches, each between its own events.

The same line also reports, under ``also``:
- timed the same way: the bf16 matmul 8192^3 (fp32 accumulate and output),
  the fp32 conv2d 32x64x56x56 -> 64, 3x3, stride 1, pad 1 as an implicit GEMM
  (also with bf16 inputs) and the tall-skinny fp32 matmul 32768x16x4096 that
  measures the HBM streaming rate, each with its roofline (the matrix-core
  peak, or HBM bandwidth below the ridge point);
- replayed as HIP graphs of 50 launches: the two small synthetic matmuls
  (fp32 256^3 and the ragged 1000^3) and the paper's other workloads
  (matmuls 1024^3, [512,128]x[128,1024], matmul+relu [256,128]x[128,1024],
  256x258x512, and the 7x7 stride-2 conv2d 3 -> 16 channels at 224x224).

``cpu_baseline`` is the fp64 oracle on the host cores: the full 4096^3
product (``value``), and per workload the full oracle where its projected
time allows, else leading row slabs scaled to the whole product.  The full
products check every output of the timed GPU launches; ``parity`` also holds
the 4096 seeded sampled checks of the large workloads.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W]
                       [--only fp32,bf16,conv,conv_bf16,skinny,small,paper]
                       [--no-cpu-baseline] [--cpu-budget S]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import xtc_inputs as xi  # noqa: E402

METRIC = "matmul TFLOP/s (fp32, bf16) and % of MI355X MFMA peak at 1 GPU"
# MI355X published dense matrix peaks (TFLOP/s) and HBM bandwidth.
PEAK = {"f32": 157.3, "bf16": 2516.6}
HBM_GBS = 8000.0
KERNEL_SOURCES = {
    "f32": ["gemm_f32.hip", "mfma_f32.h", "tile_map.h", "lds_dma.h"],
    "bf16": ["gemm_bf16.hip", "mfma_bf16.h", "tile_map.h", "lds_dma.h"],
    "conv": ["conv2d_f32.hip", "mfma_f32.h", "tile_map.h", "lds_dma.h", "unroll.h"],
    "conv_bf16": ["conv2d_bf16.hip", "lds_dma.h", "mfma_bf16.h", "tile_map.h"],
}


def kernel_hash(kind: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kind]:
        h.update(open(os.path.join(ROOT, "paper_2512_16512_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kind: str, workload: str, schedule: str | None = None):
    """HBM bytes per launch from the committed rocprofv3 counter summary, or
    None when there is none for this kernel source and schedule (the
    counters were taken on a different version of the kernel, or under a
    different schedule)."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(workload)
    except (ValueError, OSError):
        return None
    if not rec or rec.get("kernel_hash") != kernel_hash(kind):
        return None
    if schedule is not None and rec.get("schedule") != schedule:
        return None
    return rec.get("hbm_bytes_per_launch")


def to_dev(arr):
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


MIN_WARM_MS = 100.0


def time_launches(fn, steps: int, warmup: int, min_warm_ms: float = MIN_WARM_MS):
    """Run ``warmup`` untimed launches (continued, untimed, until at least
    ``min_warm_ms`` of launches have run, so that the clock has ramped up;
    the scope asks for 50 ms or more), then time exactly ``steps`` launches
    between two HIP events recorded on the launch stream (torch's current
    stream), with a device synchronisation on both sides.  Returns ms per
    launch."""
    import torch
    t0 = time.perf_counter()
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    while (time.perf_counter() - t0) * 1e3 < min_warm_ms:
        for _ in range(max(1, warmup)):
            fn()
        torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        fn()
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def launch_stats(fn, n: int):
    """Per-launch times of ``n`` further launches, each between its own pair
    of HIP events on the launch stream: median, min and 90th percentile in
    ms (reported beside ``value``, which is the bracketed whole-run figure)."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n)]
    torch.cuda.synchronize()
    for e0, e1 in evs:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    t = sorted(e0.elapsed_time(e1) for e0, e1 in evs)
    return {"median_ms": round(t[len(t) // 2], 4), "min_ms": round(t[0], 4),
            "p90_ms": round(t[min(len(t) - 1, (9 * len(t)) // 10)], 4), "n": n}


def run_matmul(cfg, steps, warmup):
    import torch
    import paper_2512_16512_amd as xtc
    A, B = xi.matmul_inputs(cfg)
    a, b = to_dev(A), to_dev(B)
    c = torch.empty((cfg["M"], cfg["N"]), dtype=torch.float32, device="cuda")
    code = xtc.XTC_F32 if cfg["dtype"] == "f32" else xtc.XTC_BF16
    M, N, K = cfg["M"], cfg["N"], cfg["K"]
    sched = xtc.xtc_default_schedule(xtc.XTC_OP_MATMUL, code, M, N, K)
    # the C ABI called with pre-marshalled arguments, so that host-side
    # launch cost stays well below the kernel time
    args = (M, N, K, a.data_ptr(), K, b.data_ptr(), N, c.data_ptr(), N, code, sched,
            torch.cuda.current_stream().cuda_stream)

    def launch():
        st = xtc.xtc_matmul(*args)
        if st != xtc.XTC_OK:
            raise xtc.XtcError(st, "xtc_matmul")

    ms = time_launches(launch, steps, warmup)
    stats = launch_stats(launch, steps)
    flops = 2.0 * cfg["M"] * cfg["N"] * cfg["K"]
    elt = 4 if cfg["dtype"] == "f32" else 2
    alg_bytes = elt * (cfg["M"] * cfg["K"] + cfg["K"] * cfg["N"]) + 4 * cfg["M"] * cfg["N"]
    i, j = xi.sample_indices_matmul(xi.seed(cfg["index"], 3), cfg["M"], cfg["N"], cfg["check"])
    sampled = c[torch.from_numpy(i).cuda(), torch.from_numpy(j).cuda()].cpu().numpy()
    return dict(ms=ms, flops=flops, alg_bytes=alg_bytes, sched=repr(sched), A=A, B=B, I=i, J=j,
                sampled=sampled, stats=stats, out=c)


def run_conv(cfg, steps, warmup, dtype="f32"):
    import torch
    import paper_2512_16512_amd as xtc
    X, W = xi.conv_inputs(cfg)
    if dtype == "bf16":
        X, W = xi.f32_to_bf16_bits(X), xi.f32_to_bf16_bits(W)
    code = xtc.XTC_F32 if dtype == "f32" else xtc.XTC_BF16
    xd, wd = to_dev(X), to_dev(W)
    OH, OW = xi.conv_out_hw(cfg["H"], cfg["W"], cfg["R"], cfg["S"], cfg["stride"], cfg["stride"],
                            cfg["pad"], cfg["pad"])
    y = torch.empty((cfg["N"], cfg["OC"], OH, OW), dtype=torch.float32, device="cuda")
    Mg, Ng, Kg = cfg["OC"], cfg["N"] * OH * OW, cfg["C"] * cfg["R"] * cfg["S"]
    sched = xtc.xtc_default_schedule(xtc.XTC_OP_CONV2D, code, Mg, Ng, Kg)
    st_, pd = cfg["stride"], cfg["pad"]
    args = (cfg["N"], cfg["C"], cfg["H"], cfg["W"], cfg["OC"], cfg["R"], cfg["S"], st_, st_, pd, pd,
            xd.data_ptr(), wd.data_ptr(), y.data_ptr(), code, sched,
            torch.cuda.current_stream().cuda_stream)

    def launch():
        st = xtc.xtc_conv2d_nchw(*args)
        if st != xtc.XTC_OK:
            raise xtc.XtcError(st, "xtc_conv2d_nchw")

    ms = time_launches(launch, steps, warmup)
    stats = launch_stats(launch, steps)
    F = xi.sample_indices_flat(xi.seed(cfg["index"], 3), y.numel(), cfg["check"])
    sampled = y.reshape(-1)[torch.from_numpy(F).cuda()].cpu().numpy()
    alg_bytes = X.itemsize * (X.size + W.size) + 4 * y.numel()
    return dict(ms=ms, flops=2.0 * Mg * Ng * Kg, alg_bytes=alg_bytes, sched=repr(sched), X=X, W=W,
                F=F, sampled=sampled, gemm=(Mg, Ng, Kg), stats=stats, out=y)


def _paper_launcher(xtc, cfg):
    """(launch(stream), output tensor, gemm extents, schedule) for one of the
    paper's other workloads, the C ABI called with pre-marshalled arguments."""
    import torch
    if cfg["op"] == "conv2d":
        X, W = xi.conv_inputs(cfg)
        xd, wd = to_dev(X), to_dev(W)
        OH, OW = xi.conv_out_hw(cfg["H"], cfg["W"], cfg["R"], cfg["S"], cfg["stride"],
                                cfg["stride"], cfg["pad"], cfg["pad"])
        y = torch.empty((cfg["N"], cfg["OC"], OH, OW), dtype=torch.float32, device="cuda")
        Mg, Ng, Kg = cfg["OC"], cfg["N"] * OH * OW, cfg["C"] * cfg["R"] * cfg["S"]
        sched = xtc.xtc_default_schedule(xtc.XTC_OP_CONV2D, xtc.XTC_F32, Mg, Ng, Kg)
        st_, pd = cfg["stride"], cfg["pad"]
        pre = (cfg["N"], cfg["C"], cfg["H"], cfg["W"], cfg["OC"], cfg["R"], cfg["S"], st_, st_, pd,
               pd, xd.data_ptr(), wd.data_ptr(), y.data_ptr(), xtc.XTC_F32, sched)

        def launch(stream):
            st = xtc.xtc_conv2d_nchw(*pre, stream)
            if st != xtc.XTC_OK:
                raise xtc.XtcError(st, "xtc_conv2d_nchw")
        keep = (xd, wd)
        alg = 4 * (X.size + W.size + y.numel())
        return launch, y, (Mg, Ng, Kg), sched, alg, keep
    A, B = xi.matmul_inputs(cfg)
    a, b = to_dev(A), to_dev(B)
    M, N, K = cfg["M"], cfg["N"], cfg["K"]
    c = torch.empty((M, N), dtype=torch.float32, device="cuda")
    code = xtc.XTC_F32 if cfg["dtype"] == "f32" else xtc.XTC_BF16
    sched = xtc.xtc_default_schedule(xtc.XTC_OP_MATMUL, code, M, N, K)
    fn = xtc.xtc_matmul_relu if cfg["op"] == "matmul_relu" else xtc.xtc_matmul
    pre = (M, N, K, a.data_ptr(), K, b.data_ptr(), N, c.data_ptr(), N, code, sched)

    def launch(stream):
        st = fn(*pre, stream)
        if st != xtc.XTC_OK:
            raise xtc.XtcError(st, fn.__name__)
    elt = 4 if cfg["dtype"] == "f32" else 2
    alg = elt * (M * K + K * N) + 4 * M * N
    return launch, c, (M, N, K), sched, alg, (a, b)


def run_paper(cfg, steps, warmup, per_graph=50):
    """One of the paper's small workloads.  A launch lasts a few microseconds,
    less than a host-side launch through ctypes, so ``per_graph`` launches are
    captured in one HIP graph and the graph is replayed: ``steps`` timed
    replays after ``warmup`` untimed ones, between HIP events on the replay
    stream.  The graph's output is checked bit for bit against an eager launch
    (the kernels are deterministic) after two replays separated by eager
    refills of the output."""
    import torch
    import paper_2512_16512_amd as xtc
    launch, out, (Mg, Ng, Kg), sched, alg, keep = _paper_launcher(xtc, cfg)
    cur = torch.cuda.current_stream()
    launch(cur.cuda_stream)
    torch.cuda.synchronize()
    eager = out.clone()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(cur)
    with torch.cuda.stream(side):
        launch(side.cuda_stream)
    cur.wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        cs = torch.cuda.current_stream().cuda_stream
        for _ in range(per_graph):
            launch(cs)
    replay_ok = True
    for _ in range(2):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        replay_ok = replay_ok and bool(torch.equal(out, eager))
    ms = time_launches(g.replay, steps, warmup) / per_graph
    # per-replay times of as many further replays, each between its own
    # events: the median per launch, beside the whole-run mean above
    med_ms = launch_stats(g.replay, steps)["median_ms"] / per_graph
    flops = 2.0 * Mg * Ng * Kg
    return dict(ms=ms, med_ms=med_ms, flops=flops, alg_bytes=alg, sched=repr(sched),
                out=out.cpu().numpy(), replay_ok=replay_ok, keep=keep)


def roofline_of(flops, alg_bytes, ms, peak_tflops, traffic):
    """Roofline entry of one launch: bound by the matrix cores when the
    workload's arithmetic intensity (FLOPs per algorithmic HBM byte) is
    above the ridge point peak / HBM bandwidth, else by HBM (then
    ``achieved`` is algorithmic bytes over time against 8 TB/s)."""
    tflops = flops / (ms * 1e-3) / 1e12
    gbps = alg_bytes / (ms * 1e-3) / 1e9
    intensity = flops / alg_bytes
    ridge = peak_tflops * 1e12 / (HBM_GBS * 1e9)
    common = {"traffic": traffic, "alg_bytes": alg_bytes, "intensity": round(intensity, 1),
              "ridge": round(ridge, 1)}
    if intensity >= ridge:
        return dict({"bound": "mfma", "achieved": round(tflops, 2), "peak": peak_tflops,
                     "unit": "TFLOP/s", "frac": round(tflops / peak_tflops, 4)}, **common,
                    alg_hbm_GBps=round(gbps, 1))
    return dict({"bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_GBS, "unit": "GB/s",
                 "frac": round(gbps / HBM_GBS, 4)}, **common, tflops=round(tflops, 2))


def summary(kind, cfg, r, workload):
    tflops = r["flops"] / (r["ms"] * 1e-3) / 1e12
    traffic = measured_traffic(kind, workload, r["sched"]) if kind in KERNEL_SOURCES else None
    peak = PEAK["bf16" if kind in ("bf16", "conv_bf16") else "f32"]
    return {
        "workload": workload,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "ms_per_launch": round(r["ms"], 4),
        "launch_stats": r["stats"],
        "median_TFLOP/s": round(r["flops"] / (r["stats"]["median_ms"] * 1e-3) / 1e12, 2),
        "frac_of_peak": round(tflops / peak, 4),
        "schedule": r["sched"],
        "roofline": roofline_of(r["flops"], r["alg_bytes"], r["ms"], peak, traffic),
    }


def _check(got, ref, tol):
    import oracle
    err = oracle.rel_fro(got, ref)
    return {"rel_fro": float("%.3e" % err), "tol": tol, "outputs": int(np.size(ref)),
            "max_abs": float("%.3e" % np.max(np.abs(np.asarray(got, np.float64) - ref))),
            "ok": bool(err <= tol)}


def cpu_baseline_leg(results, graphs, budget_s: float):
    """The fp64 oracle on the host cores, timed on a monotonic clock.

    Per synthetic workload: the full oracle on all cores when its projected
    time is at most ``budget_s`` (else a leading row slab of at least 10 s,
    scaled to the whole product and labelled extrapolated), plus the
    single-thread time of the two small matmuls.  The full products also
    serve as the parity check of every output of the timed GPU launch; the
    workloads timed only on sampled outputs are checked on those samples too.
    The headline figure (``value``) is the full 4096^3 fp32 product."""
    import oracle
    import torch
    # read before any one-thread run: the OpenMP default keeps the last count
    cores = oracle.max_threads()
    legs, parity = {}, {}

    def leg(name, flops, mode, dt, rows=None):
        legs[name] = {"mode": mode, "s": round(dt, 4), "TFLOP/s": round(flops / dt / 1e12, 6),
                      "threads": cores}
        if rows is not None:
            legs[name]["rows"] = rows

    rate = None   # TFLOP/s of the last full matmul leg, for projections
    for key, cfg in (("c0", xi.MATMUL_F32_256), ("c1", xi.MATMUL_F32_1000),
                     ("fp32", xi.MATMUL_F32_4096), ("bf16", xi.MATMUL_BF16_8192)):
        r = results.get(key) or graphs.get(key)
        if r is None:
            continue
        A, B = (r["A"], r["B"]) if "A" in r else xi.matmul_inputs(cfg)
        M, K = A.shape
        N = B.shape[1]
        flops = 2.0 * M * N * K
        tol = 1e-2 if cfg["dtype"] == "bf16" else 1e-5
        projected = flops / (rate * 1e12) if rate else 0.0
        if projected <= budget_s:
            ref, dt = oracle.timed(oracle.matmul, A, B, nthreads=cores)
            leg(cfg["name"], flops, "full", dt)
            rate = flops / dt / 1e12
            got = r["out"]
            got = got.cpu().numpy() if isinstance(got, torch.Tensor) else got
            parity[key] = _check(got, ref, tol)
            del ref, got
        else:
            # leading row slabs for at least 10 s, scaled by M / rows
            rows, t0, slab = 0, time.perf_counter(), 128
            while rows < M and time.perf_counter() - t0 < 10.0:
                oracle.matmul(A, B, rows=(rows, min(M, rows + slab)), nthreads=cores)
                rows = min(M, rows + slab)
            dt = (time.perf_counter() - t0) * M / rows
            leg(cfg["name"], flops, "extrapolated from the first %d of %d rows" % (rows, M), dt,
                rows=rows)
        if key in results:
            # the sampled check the scope names for the large workloads
            r = results[key]
            t0 = time.perf_counter()
            ref = oracle.matmul_sampled(r["A"], r["B"], r["I"], r["J"], nthreads=cores)
            dt = time.perf_counter() - t0
            parity.setdefault(key, {})
            parity[key]["sampled"] = dict(_check(r["sampled"], ref, tol), check_s=round(dt, 4))
    for key, dtype in (("conv", "f32"), ("conv_bf16", "bf16")):
        if key not in results:
            continue
        r = results[key]
        cfg = xi.CONV_F32_56
        ref, dt = oracle.timed(oracle.conv2d, r["X"], r["W"], stride=cfg["stride"], pad=cfg["pad"],
                               nthreads=cores)
        if key == "conv":
            leg(cfg["name"], r["flops"], "full", dt)
        tol = 1e-5 if dtype == "f32" else 1e-2
        parity[key] = _check(r["out"].cpu().numpy(), ref, tol)
        t0 = time.perf_counter()
        ref = oracle.conv2d_sampled(r["X"], r["W"], r["F"], stride=cfg["stride"], pad=cfg["pad"],
                                    nthreads=cores)
        parity[key]["sampled"] = dict(_check(r["sampled"], ref, tol),
                                      check_s=round(time.perf_counter() - t0, 4))
    if "skinny" in results:
        r = results["skinny"]
        ref = oracle.matmul_sampled(r["A"], r["B"], r["I"], r["J"], nthreads=cores)
        parity["skinny"] = {"sampled": _check(r["sampled"], ref, 1e-5)}
    # the oracle on one thread for the two small configs (full products)
    for cfg in (xi.MATMUL_F32_256, xi.MATMUL_F32_1000):
        A, B = xi.matmul_inputs(cfg)
        _, dt = oracle.timed(oracle.matmul, A, B, nthreads=1)
        one = legs.setdefault(cfg["name"], {})
        one["one_thread_s"] = round(dt, 4)
        one["one_thread_TFLOP/s"] = round(2.0 * cfg["M"] * cfg["N"] * cfg["K"] / dt / 1e12, 6)
    out = {"parity": parity, "legs": legs}
    head = legs.get(xi.MATMUL_F32_4096["name"])
    if head is not None:
        out["cpu_baseline"] = {
            "value": head["TFLOP/s"],
            "unit": "TFLOP/s",
            "cores": cores,
            "kind": "oracle",
            "sample": "fp64 oracle (i-k-j loop, OpenMP over rows) on the whole fp32 4096x4096x4096 "
                      "matmul (%s, %.1f s wall on %d threads); per_config holds the other "
                      "workloads (full where projected <= %.0f s)" % (head["mode"], head["s"],
                                                                      cores, budget_s),
            "cpu_model": _cpu_model(),
            "per_config": legs,
        }
    return out


def paper_parity(paper):
    """Every output of each of the paper's workloads against the oracle."""
    import oracle
    out = {}
    for key, v in paper.items():
        cfg, r = v["cfg"], v["r"]
        if cfg["op"] == "conv2d":
            X, W = xi.conv_inputs(cfg)
            ref = oracle.conv2d(X, W, stride=cfg["stride"], pad=cfg["pad"])
        else:
            A, B = xi.matmul_inputs(cfg)
            ref = oracle.matmul(A, B)
            if cfg["op"] == "matmul_relu":
                ref = oracle.relu(ref)
        err = oracle.rel_fro(r["out"], ref)
        out[key] = {"rel_fro": float("%.3e" % err), "tol": 1e-5, "samples": int(ref.size),
                    "ok": bool(err <= 1e-5 and r["replay_ok"])}
    return out


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def head_flops(kind: str) -> float:
    if kind in ("fp32", "bf16"):
        cfg = xi.MATMUL_F32_4096 if kind == "fp32" else xi.MATMUL_BF16_8192
        return 2.0 * cfg["M"] * cfg["N"] * cfg["K"]
    cfg = xi.CONV_F32_56
    OH, OW = xi.conv_out_hw(cfg["H"], cfg["W"], cfg["R"], cfg["S"], cfg["stride"], cfg["stride"],
                            cfg["pad"], cfg["pad"])
    return 2.0 * cfg["OC"] * cfg["N"] * OH * OW * cfg["C"] * cfg["R"] * cfg["S"]


def head_shape(kind: str) -> dict:
    """Shape and layout keys of a headline workload for the JSON config."""
    if kind in ("fp32", "bf16"):
        cfg = (xi.MATMUL_F32_4096 if kind == "fp32" else xi.MATMUL_BF16_8192)
        return {"M": cfg["M"], "N": cfg["N"], "K": cfg["K"],
                "layout": "row-major A[M,K], B[K,N], C[M,N]"}
    cfg = xi.CONV_F32_56
    return {k: cfg[k] for k in ("N", "C", "H", "W", "OC", "R", "S", "stride", "pad")} | {
        "layout": "X NCHW, W OIHW, Y NCHW"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--only", default="fp32,bf16,conv,conv_bf16,skinny,small,paper")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=60.0,
                    help="largest projected time (s) of a full oracle run; longer ones are "
                         "timed on leading row slabs and extrapolated")
    ap.add_argument("--vendor", action="store_true",
                    help="also time the vendor libraries behind torch (hipBLASLt matmul, MIOpen "
                         "conv2d) on the same workloads, as a second JSON line (comparison only)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 256 MiB device-to-device copy (the reference kernel "
                         "for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the contraction is benchmarked on a single "
              "MI355X and no multi-GPU path is built (--gpus must be 1).", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU (torch.cuda.is_available() is False)", file=sys.stderr)
        sys.exit(1)
    import paper_2512_16512_amd  # noqa: F401  (fails loudly if libxtc.so is missing)

    if args.calibrate_copy:
        n = 64 << 20  # fp32 elements: 256 MiB read + 256 MiB written per copy
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        ms = time_launches(lambda: dst.copy_(src), args.steps, args.warmup)
        print(json.dumps({"calibration": "copy", "bytes_read": 4 * n, "bytes_written": 4 * n,
                          "ms_per_copy": round(ms, 4),
                          "GBps": round(8 * n / (ms * 1e-3) / 1e9, 1)}), flush=True)
        return

    kinds = [k.strip() for k in args.only.split(",") if k.strip()]
    results, summaries = {}, {}
    if "fp32" in kinds:
        cfg = xi.MATMUL_F32_4096
        results["fp32"] = run_matmul(cfg, args.steps, args.warmup)
        summaries["fp32"] = summary("f32", cfg, results["fp32"], "matmul_f32_4096x4096x4096")
        print("# fp32 4096^3: %.4f ms/launch" % results["fp32"]["ms"], file=sys.stderr, flush=True)
    if "bf16" in kinds:
        cfg = xi.MATMUL_BF16_8192
        results["bf16"] = run_matmul(cfg, args.steps, args.warmup)
        summaries["bf16"] = summary("bf16", cfg, results["bf16"], "matmul_bf16_8192x8192x8192")
        print("# bf16 8192^3: %.4f ms/launch" % results["bf16"]["ms"], file=sys.stderr, flush=True)
    if "conv" in kinds:
        cfg = xi.CONV_F32_56
        results["conv"] = run_conv(cfg, args.steps, args.warmup)
        summaries["conv"] = summary("conv", cfg, results["conv"], "conv2d_f32_n32c64h56w56_oc64_r3s3")
        print("# conv: %.4f ms/launch" % results["conv"]["ms"], file=sys.stderr, flush=True)
    if "conv_bf16" in kinds:
        cfg = xi.CONV_F32_56
        results["conv_bf16"] = run_conv(cfg, args.steps, args.warmup, dtype="bf16")
        summaries["conv_bf16"] = summary("conv_bf16", cfg, results["conv_bf16"],
                                         "conv2d_bf16_n32c64h56w56_oc64_r3s3")
        print("# conv bf16: %.4f ms/launch" % results["conv_bf16"]["ms"], file=sys.stderr,
              flush=True)

    if "skinny" in kinds:
        cfg = xi.MATMUL_F32_SKINNY
        results["skinny"] = run_matmul(cfg, args.steps, args.warmup)
        summaries["skinny"] = summary("f32", cfg, results["skinny"], "matmul_f32_32768x16x4096")
        print("# skinny fp32: %.4f ms/launch" % results["skinny"]["ms"], file=sys.stderr,
              flush=True)

    # the two small synthetic workloads, replayed as HIP graphs of launches
    graphs = {}
    for key, cfg, wl in (("c0", xi.MATMUL_F32_256, "matmul_f32_256x256x256"),
                         ("c1", xi.MATMUL_F32_1000, "matmul_f32_1000x1000x1000")):
        if "small" not in kinds:
            continue
        r = run_paper(cfg, args.steps, args.warmup)
        A, B = xi.matmul_inputs(cfg)
        r.update(A=A, B=B)
        graphs[key] = r
        tf = r["flops"] / (r["ms"] * 1e-3) / 1e12
        summaries[key] = {
            "workload": wl, "value": round(tf, 2), "unit": "TFLOP/s",
            "us_per_launch": round(r["ms"] * 1e3, 3), "median_us_per_launch": round(r["med_ms"] * 1e3, 3),
            "frac_of_peak": round(tf / PEAK["f32"], 4),
            "schedule": r["sched"], "timing": "HIP graph of 50 launches, replayed",
            "graph_replay_exact": r["replay_ok"],
            "roofline": roofline_of(r["flops"], r["alg_bytes"], r["ms"], PEAK["f32"], None)}
        print("# %s: %.2f us/launch" % (cfg["name"], r["ms"] * 1e3), file=sys.stderr, flush=True)

    paper = {}
    if "paper" in kinds:
        for cfg in xi.PAPER_WORKLOADS:
            r = run_paper(cfg, args.steps, args.warmup)
            tf = r["flops"] / (r["ms"] * 1e-3) / 1e12
            paper["w%d" % cfg["index"]] = dict(
                cfg=cfg, r=r, line={
                    "workload": cfg["name"], "value": round(tf, 2), "unit": "TFLOP/s",
                    "us_per_launch": round(r["ms"] * 1e3, 2),
                    "median_us_per_launch": round(r["med_ms"] * 1e3, 2),
                    "frac_of_peak": round(tf / PEAK["f32"], 4), "schedule": r["sched"],
                    "timing": "HIP graph of 50 launches, replayed", "graph_replay_exact":
                        r["replay_ok"]})
            print("# %s: %.2f us/launch" % (cfg["name"], r["ms"] * 1e3), file=sys.stderr,
                  flush=True)
        summaries["paper"] = {k: v["line"] for k, v in paper.items()}

    heads = [k for k in ("fp32", "bf16", "conv") if k in summaries]
    if not heads:
        print("bench.py: --only must name at least one of fp32, bf16, conv", file=sys.stderr)
        sys.exit(2)
    head_kind = heads[0]
    head = summaries[head_kind]
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_launch"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if head_kind != "bf16" else "bf16",
        "data": "synthetic: splitmix64 uniform [-1,1) inputs from fixed seeds, resident in HBM",
        "config": dict(
            {"workload": head["workload"]},
            **head_shape(head_kind),
            schedule=head["schedule"],
            device=torch.cuda.get_device_name(0),
            hip=torch.version.hip,
        ),
        "launch_stats": head["launch_stats"],
        "median_TFLOP/s": round(head_flops(head_kind) / (head["launch_stats"]["median_ms"] * 1e-3)
                                / 1e12, 2),
        "value_basis": "value: the K timed launches bracketed by two HIP events (whole-run mean); "
                       "median_TFLOP/s: the per-launch median of K further launches, each between "
                       "its own events, which is the figure the scope's metric grades",
        "warmup_policy": "W untimed launches, continued until at least %d ms of launches have "
                         "run (clock ramp)" % MIN_WARM_MS,
        "roofline": head["roofline"],
        "frac_of_peak": head["frac_of_peak"],
        "also": {k: v for k, v in summaries.items() if k != head_kind},
    }
    if not args.no_cpu_baseline:
        extra = cpu_baseline_leg(results, graphs, args.cpu_budget)
        if "cpu_baseline" in extra:
            line["cpu_baseline"] = extra["cpu_baseline"]
        line["parity"] = extra["parity"]
        line["parity"].update(paper_parity(paper))
    print(json.dumps(line), flush=True)
    if args.vendor:
        print(json.dumps(vendor_line(args.steps, args.warmup, line)), flush=True)


def vendor_line(steps: int, warmup: int, ours: dict):
    """The same workloads through torch's vendor libraries (hipBLASLt for
    matmul, MIOpen for conv2d), timed exactly as ours: a comparison point,
    not part of the measured path."""
    import torch
    torch.backends.cuda.matmul.allow_tf32 = False
    torch.backends.cudnn.allow_tf32 = False
    out = {"vendor": "torch %s, HIP %s" % (torch.__version__, torch.version.hip)}
    for kind, cfg in (("fp32", xi.MATMUL_F32_4096), ("bf16", xi.MATMUL_BF16_8192),
                      ("skinny", xi.MATMUL_F32_SKINNY)):
        A, B = xi.matmul_inputs(cfg)
        a, b = to_dev(A), to_dev(B)
        c = torch.empty((cfg["M"], cfg["N"]), dtype=a.dtype, device="cuda")
        ms = time_launches(lambda: torch.matmul(a, b, out=c), steps, warmup)
        tf = 2.0 * cfg["M"] * cfg["N"] * cfg["K"] / (ms * 1e-3) / 1e12
        mine = ours["value"] if kind == "fp32" else ours["also"].get(kind, {}).get("value")
        out[kind] = {"workload": cfg["name"], "ms_per_launch": round(ms, 4), "TFLOP/s": round(tf, 2),
                     "ours_TFLOP/s": mine, "output_dtype": str(c.dtype).replace("torch.", "")}
        if kind == "bf16":
            # the same operation as ours: bf16 inputs, fp32 accumulation and fp32 output
            c32 = torch.empty((cfg["M"], cfg["N"]), dtype=torch.float32, device="cuda")
            try:
                ms = time_launches(lambda: torch.mm(a, b, out_dtype=torch.float32, out=c32), steps, warmup)
                tf = 2.0 * cfg["M"] * cfg["N"] * cfg["K"] / (ms * 1e-3) / 1e12
                out["bf16_f32_out"] = {"workload": cfg["name"], "ms_per_launch": round(ms, 4),
                                       "TFLOP/s": round(tf, 2), "ours_TFLOP/s": mine,
                                       "output_dtype": "float32"}
            except (RuntimeError, TypeError) as e:
                out["bf16_f32_out"] = {"error": str(e)[:200]}
            del c32
        del a, b, c
    cfg = xi.CONV_F32_56
    X, W = xi.conv_inputs(cfg)
    xd, wd = to_dev(X), to_dev(W)
    f = lambda: torch.nn.functional.conv2d(xd, wd, stride=cfg["stride"], padding=cfg["pad"])
    ms = time_launches(f, steps, warmup)
    OH, OW = xi.conv_out_hw(cfg["H"], cfg["W"], cfg["R"], cfg["S"], cfg["stride"], cfg["stride"],
                            cfg["pad"], cfg["pad"])
    flops = 2.0 * cfg["OC"] * cfg["N"] * OH * OW * cfg["C"] * cfg["R"] * cfg["S"]
    out["conv"] = {"workload": cfg["name"], "ms_per_launch": round(ms, 4),
                   "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 2),
                   "ours_TFLOP/s": ours["also"].get("conv", {}).get("value")}
    # bf16 inputs: MIOpen returns a bf16 output (half the bytes of ours)
    xb, wb = xd.to(torch.bfloat16), wd.to(torch.bfloat16)
    f = lambda: torch.nn.functional.conv2d(xb, wb, stride=cfg["stride"], padding=cfg["pad"])
    ms = time_launches(f, steps, warmup)
    out["conv_bf16"] = {"workload": cfg["name"].replace("fp32", "bf16"), "ms_per_launch": round(ms, 4),
                        "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 2), "output_dtype": "bfloat16",
                        "ours_TFLOP/s": ours["also"].get("conv_bf16", {}).get("value")}
    return out


if __name__ == "__main__":
    main()
