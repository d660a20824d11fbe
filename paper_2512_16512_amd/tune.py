"""Schedule exploration over the compiled design space.

The GPU counterpart of the paper's exploration strategies (Sec. 5.2): a
strategy names a design space of schedules for one operator, draws samples
from it, applies each sample to the operator, and compiles and evaluates the
result; ``default_schedule`` gives one good point without a search.  Here the
design space is the product of the kernel instances compiled into
``libxtc.so`` (tile sizes, wave tiles, MFMA shape, LDS ring depth, layout and
reduction order: the compile-time primitives) with the two run-time
interchange choices, the tile raster order and the XCD remap.  Each sample is
evaluated as the paper's harness does (Sec. 4.2): run on the device, its
output validated against a reference output, then timed.  The reference is
the output of the library's default schedule for the same inputs; a sample
whose output differs from it by more than the dtype's tolerance is reported
as invalid and never ranked.

Timing: a launch of a small problem lasts a few microseconds, less than the
host-side cost of a launch, so ``per_graph`` launches are captured in one HIP
graph and the graph is replayed; the time per launch is the event time of
the replays divided by the launches they contain.

Usage::

    python -m paper_2512_16512_amd.tune matmul f32 1024 1024 1024 [--samples 40] [--journal f.jsonl]
    python -m paper_2512_16512_amd.tune conv2d f32 1 3 224 224 16 7 7 2 3
"""
from __future__ import annotations

import argparse
import json
import random
import sys

import paper_2512_16512_amd as xtc

RASTERS = (0, 1, 4, 8, 16)
TOL = {"f32": 1e-5, "bf16": 1e-2}


class Problem:
    """One operator instance with device-resident seeded inputs.

    ``op`` is "matmul", "matmul_relu", "conv2d" or "conv2d_relu"; ``dims`` is
    (M, N, K) for a matmul and (N, C, H, W, OC, R, S, stride, pad) for a
    conv2d.  Inputs are uniform in [-1, 1) from a fixed torch generator."""

    def __init__(self, op: str, dtype: str, dims, seed: int = 0):
        import torch
        self.op, self.dtype, self.dims = op, dtype, tuple(int(d) for d in dims)
        self.relu = op.endswith("_relu")
        self.is_conv = op.startswith("conv2d")
        if dtype not in ("f32", "bf16"):
            raise ValueError("dtype must be f32 or bf16")
        self.code = xtc.XTC_F32 if dtype == "f32" else xtc.XTC_BF16
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16

        def rnd(*shape):
            return (torch.rand(shape, generator=g, device="cuda") * 2 - 1).to(tdt).contiguous()

        if self.is_conv:
            if len(self.dims) != 9:
                raise ValueError("conv2d dims: N C H W OC R S stride pad")
            N, C, H, W, OC, R, S, st, pd = self.dims
            self.x, self.w = rnd(N, C, H, W), rnd(OC, C, R, S)
            OH, OW = (H + 2 * pd - R) // st + 1, (W + 2 * pd - S) // st + 1
            self.out = torch.empty((N, OC, OH, OW), dtype=torch.float32, device="cuda")
            self.gemm = (OC, N * OH * OW, C * R * S)
            self.op_code = xtc.XTC_OP_CONV2D
            self._fn = xtc.xtc_conv2d_nchw_relu if self.relu else xtc.xtc_conv2d_nchw
            self._pre = (N, C, H, W, OC, R, S, st, st, pd, pd, self.x.data_ptr(),
                         self.w.data_ptr(), self.out.data_ptr(), self.code)
        else:
            if len(self.dims) != 3:
                raise ValueError("matmul dims: M N K")
            M, N, K = self.dims
            self.a, self.b = rnd(M, K), rnd(K, N)
            self.out = torch.empty((M, N), dtype=torch.float32, device="cuda")
            self.gemm = (M, N, K)
            self.op_code = xtc.XTC_OP_MATMUL
            self._fn = xtc.xtc_matmul_relu if self.relu else xtc.xtc_matmul
            self._pre = (M, N, K, self.a.data_ptr(), K, self.b.data_ptr(), N,
                         self.out.data_ptr(), N, self.code)

    @property
    def flops(self) -> float:
        M, N, K = self.gemm
        return 2.0 * M * N * K

    def launch(self, sched, stream: int) -> None:
        st = self._fn(*self._pre, sched, stream)
        if st != xtc.XTC_OK:
            raise xtc.XtcError(st, self._fn.__name__)

    def default_schedule(self):
        M, N, K = self.gemm
        return xtc.xtc_default_schedule(self.op_code, self.code, M, N, K)

    def __repr__(self):
        return "%s %s %s" % (self.op, self.dtype, "x".join(str(d) for d in self.dims))


def design_space(op_code: int, dtype_code: int, rasters=RASTERS, xcd=(0, 1)):
    """Every compiled instance for op/dtype crossed with the run-time raster
    orders and XCD remaps."""
    out = []
    for s in xtc.xtc_sched_list(op_code, dtype_code):
        for r in rasters:
            for x in xcd:
                t = xtc.Sched(**s.as_dict())
                t.raster, t.xcd_remap = r, x
                out.append(t)
    return out


def sample(space, n: int, seed: int = 0):
    """``n`` distinct points of ``space`` drawn with a seeded generator (all of
    them, in a seeded order, when ``n`` >= the size of the space)."""
    idx = list(range(len(space)))
    random.Random(seed).shuffle(idx)
    return [space[i] for i in idx[:n]]


def _rel_fro(got, ref) -> float:
    import torch
    den = torch.linalg.vector_norm(ref.double())
    num = torch.linalg.vector_norm((got.double() - ref.double()))
    if float(den) == 0.0:
        return 0.0 if float(num) == 0.0 else float("inf")
    return float(num / den)


def evaluate(problem: Problem, sched, reference=None, per_graph: int = 0, replays: int = 10,
             warmup: int = 2):
    """Run, validate and time one schedule.  Returns a dict with ``us`` (time
    per launch), ``tflops``, ``err`` (relative Frobenius distance to
    ``reference``, if given) and ``valid``."""
    import torch
    cur = torch.cuda.current_stream()
    problem.out.fill_(float("nan"))
    problem.launch(sched, cur.cuda_stream)
    torch.cuda.synchronize()
    err = _rel_fro(problem.out, reference) if reference is not None else 0.0
    valid = bool(torch.isfinite(problem.out).all()) and err <= TOL[problem.dtype]
    # size the graph from one eager launch: about 2 ms of device time per replay
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    problem.launch(sched, cur.cuda_stream)
    t1.record()
    torch.cuda.synchronize()
    if per_graph <= 0:
        per_graph = int(min(100, max(1, 2.0 / max(t0.elapsed_time(t1), 1e-3))))
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(cur)
    with torch.cuda.stream(side):
        problem.launch(sched, side.cuda_stream)
    cur.wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        cs = torch.cuda.current_stream().cuda_stream
        for _ in range(per_graph):
            problem.launch(sched, cs)
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    t0.record()
    for _ in range(replays):
        g.replay()
    t1.record()
    torch.cuda.synchronize()
    us = t0.elapsed_time(t1) * 1e3 / (replays * per_graph)
    del g
    return {"us": us, "tflops": problem.flops / (us * 1e-6) / 1e12, "err": err, "valid": valid,
            "per_graph": per_graph}


def warm_up(problem: Problem, sched, ms: float = 100.0) -> None:
    """Launch ``sched`` for about ``ms`` milliseconds so that the first timed
    evaluation does not run on a cold (lower-clocked) GPU."""
    import time

    import torch
    stream = torch.cuda.current_stream().cuda_stream
    t0 = time.perf_counter()
    while (time.perf_counter() - t0) * 1e3 < ms:
        for _ in range(10):
            problem.launch(sched, stream)
        torch.cuda.synchronize()


def _key(sched) -> str:
    return json.dumps(sched.as_dict(), sort_keys=True)


def read_journal(path: str, problem_key: str) -> dict:
    """Results already recorded in the JSON-lines journal ``path`` for the
    problem ``problem_key``, by schedule (an incomplete last line, left by an
    interrupted run, is ignored)."""
    done = {}
    try:
        lines = open(path).read().splitlines()
    except FileNotFoundError:
        return done
    for line in lines:
        try:
            rec = json.loads(line)
        except ValueError:
            continue
        if rec.get("problem") == problem_key:
            done[json.dumps(rec["sched"], sort_keys=True)] = rec
    return done


def explore(problem: Problem, n: int | None = None, seed: int = 0, space=None, log=None,
            journal: str | None = None):
    """Evaluate ``n`` sampled schedules (the whole design space when None),
    plus the default schedule, against the default schedule's output.
    Returns (default result, results sorted fastest first).

    With ``journal`` (a JSON-lines file), every evaluated point is appended
    to it as soon as it is measured, and points the journal already holds for
    this problem are taken from it instead of being run again: an
    interrupted sweep resumes where it stopped."""
    if space is None:
        space = design_space(problem.op_code, problem.code)
    pts = space if n is None else sample(space, n, seed)
    dflt = problem.default_schedule()
    warm_up(problem, dflt)
    base = evaluate(problem, dflt)
    reference = problem.out.clone()
    base["sched"] = dflt
    pkey = repr(problem)
    done = read_journal(journal, pkey) if journal else {}
    results = []
    for s in pts:
        rec = done.get(_key(s))
        if rec is not None:
            r = {k: v for k, v in rec.items() if k not in ("problem", "sched")}
        else:
            r = evaluate(problem, s, reference)
            if journal:
                with open(journal, "a") as f:
                    f.write(json.dumps(dict({"problem": pkey, "sched": s.as_dict()}, **r)) + "\n")
        r["sched"] = s
        results.append(r)
        if log:
            log("%-100r %9.2f us %8.2f TF err %.1e%s%s" % (
                s, r["us"], r["tflops"], r["err"], "" if r["valid"] else "  INVALID",
                "  (journal)" if rec is not None else ""))
    results.sort(key=lambda r: (not r["valid"], r["us"]))
    return base, results


def _as_json(r):
    d = {k: v for k, v in r.items() if k != "sched"}
    d["sched"] = r["sched"].as_dict()
    return d


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("op", choices=["matmul", "matmul_relu", "conv2d", "conv2d_relu"])
    ap.add_argument("dtype", choices=["f32", "bf16"])
    ap.add_argument("dims", type=int, nargs="+")
    ap.add_argument("--samples", type=int, default=None, help="sampled points (default: all)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--json", default=None, help="write every result to this file")
    ap.add_argument("--journal", default=None,
                    help="JSON-lines file: append each point as it is measured and skip points "
                         "already recorded for this problem (resumes an interrupted sweep)")
    ap.add_argument("--quiet", action="store_true")
    a = ap.parse_args(argv)
    p = Problem(a.op, a.dtype, a.dims)
    log = None if a.quiet else (lambda s: print(s, flush=True))
    base, res = explore(p, a.samples, a.seed, log=log, journal=a.journal)
    best = res[0]
    print("problem  %r" % p)
    print("default  %r  %.2f us  %.2f TFLOP/s" % (base["sched"], base["us"], base["tflops"]))
    print("best     %r  %.2f us  %.2f TFLOP/s  (%.2fx the default)" % (
        best["sched"], best["us"], best["tflops"], base["us"] / best["us"]))
    print("invalid  %d of %d" % (sum(not r["valid"] for r in res), len(res)), flush=True)
    if a.json:
        with open(a.json, "w") as f:
            json.dump({"problem": repr(p), "default": _as_json(base),
                       "results": [_as_json(r) for r in res]}, f, indent=1)
    return 0 if all(r["valid"] for r in res) else 1


if __name__ == "__main__":
    sys.exit(main())
