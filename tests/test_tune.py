"""Schedule exploration (paper_2512_16512_amd.tune): the design space and its
seeded sampling on the CPU; a small exploration on the GPU, where every
sampled schedule must validate against the default schedule's output."""
import pytest


@pytest.fixture(scope="module")
def t():
    from paper_2512_16512_amd import tune
    return tune


def test_design_space_is_compiled_instances_times_runtime_choices(t):
    import paper_2512_16512_amd as x
    for op, dt in ((x.XTC_OP_MATMUL, x.XTC_F32), (x.XTC_OP_MATMUL, x.XTC_BF16),
                   (x.XTC_OP_CONV2D, x.XTC_F32)):
        space = t.design_space(op, dt)
        n_inst = len(x.xtc_sched_list(op, dt))
        assert len(space) == n_inst * len(t.RASTERS) * 2
        keys = {tuple(sorted(s.as_dict().items())) for s in space}
        assert len(keys) == len(space)
        for s in space:
            assert x.xtc_sched_check(op, dt, s) == 0


def test_sample_is_seeded_and_distinct(t):
    import paper_2512_16512_amd as x
    space = t.design_space(x.XTC_OP_MATMUL, x.XTC_F32)
    a = t.sample(space, 12, seed=3)
    b = t.sample(space, 12, seed=3)
    c = t.sample(space, 12, seed=4)
    key = lambda s: tuple(sorted(s.as_dict().items()))  # noqa: E731
    assert [key(s) for s in a] == [key(s) for s in b]
    assert [key(s) for s in a] != [key(s) for s in c]
    assert len({key(s) for s in a}) == 12
    assert len(t.sample(space, 10 ** 6)) == len(space)


def test_journal_resumes_an_interrupted_sweep(t, tmp_path, monkeypatch):
    """Host logic of the sweep journal, with the measurement replaced by a
    deterministic stand-in: points are appended as they are measured, a
    second run over the same journal measures nothing, a run cut short
    resumes with only the missing points, and an incomplete last line or
    another problem's lines are not taken as results."""
    import json

    import paper_2512_16512_amd as x
    space = t.design_space(x.XTC_OP_MATMUL, x.XTC_F32)[:9]
    calls = []

    def fake_evaluate(problem, sched, reference=None, **kw):
        calls.append(t._key(sched))
        us = 1.0 + sched.block_m / 64.0 + sched.raster + 0.5 * sched.xcd_remap
        return {"us": us, "tflops": 1.0 / us, "err": 0.0, "valid": True, "per_graph": 1}

    class FakeOut:
        def clone(self):
            return self

    class FakeProblem:
        op_code, code, out = x.XTC_OP_MATMUL, x.XTC_F32, FakeOut()

        def __init__(self, name):
            self.name = name

        def default_schedule(self):
            return space[0]

        def __repr__(self):
            return self.name

    monkeypatch.setattr(t, "evaluate", fake_evaluate)
    monkeypatch.setattr(t, "warm_up", lambda p, s, ms=0: None)
    j = str(tmp_path / "sweep.jsonl")
    _, full = t.explore(FakeProblem("p"), space=space, journal=j)
    assert len(calls) == 1 + 9 and len(open(j).read().splitlines()) == 9
    calls.clear()
    _, again = t.explore(FakeProblem("p"), space=space, journal=j)
    assert len(calls) == 1                       # only the default's reference run
    assert [r["us"] for r in again] == [r["us"] for r in full]
    # cut short after 4 points, with a torn fifth line and another problem's line
    lines = open(j).read().splitlines()
    other = json.loads(lines[5])
    other["problem"] = "q"
    open(j, "w").write("\n".join(lines[:4] + [json.dumps(other), lines[4][:20]]))
    calls.clear()
    _, resumed = t.explore(FakeProblem("p"), space=space, journal=j)
    assert sorted(calls[1:]) == sorted(t._key(s) for s in space[4:])
    assert [r["us"] for r in resumed] == [r["us"] for r in full]


@pytest.mark.gpu
@pytest.mark.parametrize("op,dtype,dims", [
    ("matmul", "f32", (200, 300, 96)),
    ("matmul_relu", "bf16", (130, 260, 64)),
    ("conv2d", "f32", (1, 3, 40, 40, 16, 7, 7, 2, 3)),
    ("conv2d_relu", "bf16", (2, 16, 20, 20, 24, 3, 3, 1, 1)),
])
def test_explore_small_problem(t, op, dtype, dims):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    p = t.Problem(op, dtype, dims, seed=1)
    print("[gpu] explore", p, flush=True)
    base, res = t.explore(p, n=8, seed=0)
    assert base["valid"] and base["us"] > 0
    assert len(res) == 8 and all(r["valid"] for r in res), [r["err"] for r in res]
    assert res[0]["us"] <= res[-1]["us"]
