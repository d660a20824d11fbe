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
