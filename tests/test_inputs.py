"""Seeded input generator: published test vectors, exactness, bf16 rounding."""
import json
import os

import numpy as np
import torch

import xtc_inputs as xi

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_splitmix64_published_vector():
    g = json.load(open(os.path.join(GOLDEN, "splitmix64_seed0.json")))
    got = xi.splitmix64(g["seed"], 3)
    assert [format(int(v), "016x") for v in got] == g["outputs_hex"]


def test_splitmix64_counter_offsets():
    full = xi.splitmix64(77, 3 * (1 << 20) + 5)          # crosses chunk borders
    part = xi.splitmix64(77, 1000, start=(1 << 20) - 10)
    assert np.array_equal(full[(1 << 20) - 10:(1 << 20) + 990], part)


def test_uniform_range_grid_and_exactness():
    a = xi.uniform_f32(1, (1 << 16,))
    assert a.dtype == np.float32
    assert a.min() >= -1.0 and a.max() < 1.0
    scaled = (a.astype(np.float64) + 1.0) * 2.0 ** 23
    assert np.array_equal(scaled, np.round(scaled))  # on the 2**-23 grid
    # the same value computed in fp64 from the raw stream
    z = xi.splitmix64(1, 1 << 16)
    ref = (z >> np.uint64(40)).astype(np.float64) * 2.0 ** -23 - 1.0
    assert np.array_equal(a.astype(np.float64), ref)
    # roughly uniform
    assert abs(float(a.mean())) < 0.02


def test_uniform_is_deterministic_and_seed_dependent():
    a = xi.uniform_f32(2001, (64, 64))
    b = xi.uniform_f32(2001, (64, 64))
    c = xi.uniform_f32(2002, (64, 64))
    assert np.array_equal(a, b)
    assert not np.array_equal(a, c)


def test_bf16_rounding_matches_torch():
    x = xi.uniform_f32(5, (1 << 18,))
    # add values exactly halfway between two bf16 numbers (ties to even)
    ties = np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -1.0 - 2.0 ** -8, 0.5 + 2.0 ** -9],
                    dtype=np.float32)
    x = np.concatenate([x, ties])
    ours = xi.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    # ties: 1 + 2^-8 rounds down to 1.0 (even), 1 + 3*2^-8 rounds up to 1 + 2^-6
    assert ours[-4] == 0x3F80 and ours[-3] == 0x3F82


def test_bf16_widening_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3FC0, 0x0000, 0x8000, 0x4049], dtype=np.uint16)
    f = xi.bf16_bits_to_f32(bits)
    assert f.tolist()[:5] == [1.0, -2.0, 1.5, 0.0, -0.0]
    assert abs(f[5] - 3.140625) == 0.0


def test_small_int_range():
    a = xi.small_int_f32(9, (4096,))
    assert set(np.unique(a).tolist()) == {-2.0, -1.0, 0.0, 1.0, 2.0}


def test_sample_indices():
    i, j = xi.sample_indices_matmul(2003, 4096, 4096)
    assert i.shape == (4096,) and j.shape == (4096,)
    assert i.min() >= 0 and i.max() < 4096 and j.min() >= 0 and j.max() < 4096
    z = xi.splitmix64(2003, 4096)
    assert int(i[0]) == int(z[0] >> np.uint64(32)) % 4096
    assert int(j[0]) == int(z[0] & np.uint64(0xFFFFFFFF)) % 4096
    f = xi.sample_indices_flat(4003, 32 * 64 * 56 * 56)
    assert f.min() >= 0 and f.max() < 32 * 64 * 56 * 56


def test_workload_shapes():
    c = xi.WORKLOADS
    assert [x["index"] for x in c] == [0, 1, 2, 3, 4]
    assert (xi.MATMUL_F32_256, xi.MATMUL_F32_1000, xi.MATMUL_F32_4096, xi.MATMUL_BF16_8192,
            xi.CONV_F32_56) == tuple(c)
    assert (c[3]["M"], c[3]["dtype"]) == (8192, "bf16")
    oh, ow = xi.conv_out_hw(56, 56, 3, 3, 1, 1, 1, 1)
    assert (oh, ow) == (56, 56)
    sk = xi.MATMUL_F32_SKINNY
    assert sk["index"] not in {x["index"] for x in c + xi.PAPER_WORKLOADS}   # distinct seeds
    # below the fp32 ridge point (157.3 TFLOP/s over 8 TB/s = 19.7 FLOP per byte)
    fl = 2.0 * sk["M"] * sk["N"] * sk["K"]
    by = 4 * (sk["M"] * sk["K"] + sk["K"] * sk["N"] + sk["M"] * sk["N"])
    assert fl / by < 19.7


def test_paper_workload_shapes():
    w = {c["index"]: c for c in xi.PAPER_WORKLOADS}
    assert sorted(w) == [5, 6, 7, 8, 9]
    assert (w[6]["M"], w[6]["K"], w[6]["N"]) == (512, 128, 1024)
    assert (w[7]["M"], w[7]["K"], w[7]["N"], w[7]["op"]) == (256, 128, 1024, "matmul_relu")
    assert (w[8]["M"], w[8]["N"], w[8]["K"]) == (256, 258, 512)
    c = w[9]
    oh, ow = xi.conv_out_hw(c["H"], c["W"], c["R"], c["S"], c["stride"], c["stride"], c["pad"],
                            c["pad"])
    assert (oh, ow, c["OC"], c["C"]) == (112, 112, 16, 3)     # [112,112,16] x [7,7,3]
    assert not set(w) & {x["index"] for x in xi.WORKLOADS}        # distinct seeds
