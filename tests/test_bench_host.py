"""Host-side logic of bench.py that needs no GPU: the one-GPU rule and the
rule that measured traffic is reported only for the kernel sources it was
measured on."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_only_for_the_measured_kernel_source(monkeypatch):
    import json
    path = os.path.join(ROOT, "profiles", "traffic.json")
    rec = json.load(open(path))
    for workload, kind in (("matmul_f32_4096x4096x4096", "f32"),
                           ("matmul_bf16_8192x8192x8192", "bf16"),
                           ("conv2d_f32_n32c64h56w56_oc64_r3s3", "conv"),
                           ("matmul_f32_32768x16x4096", "f32"),
                           ("conv2d_bf16_n32c64h56w56_oc64_r3s3", "conv_bf16")):
        assert workload in rec
        monkeypatch.setattr(bench, "kernel_hash", lambda k: rec[workload]["kernel_hash"])
        assert bench.measured_traffic(kind, workload) == rec[workload]["hbm_bytes_per_launch"]
        if "schedule" in rec[workload]:
            assert bench.measured_traffic(kind, workload, rec[workload]["schedule"]) == \
                rec[workload]["hbm_bytes_per_launch"]
            assert bench.measured_traffic(kind, workload, "another schedule") is None
        monkeypatch.setattr(bench, "kernel_hash", lambda k: "0" * 16)
        assert bench.measured_traffic(kind, workload) is None


def test_kernel_hash_covers_every_source_of_the_kernel():
    import re
    csrc = os.path.join(ROOT, "paper_2512_16512_amd", "csrc")
    for kind, files in bench.KERNEL_SOURCES.items():
        for f in files:
            assert os.path.exists(os.path.join(csrc, f))
        # every kernel header the kernel's source includes is hashed too
        inc = set(re.findall(r'#include "([a-z_0-9]+\.h)"', open(os.path.join(csrc, files[0])).read()))
        assert inc - {"xtc_internal.h"} <= set(files), (kind, inc - set(files))
        assert bench.kernel_hash(kind) == bench.kernel_hash(kind)


def test_roofline_bound_follows_the_ridge_point():
    """A workload whose FLOPs per algorithmic HBM byte fall below peak / 8 TB/s
    is reported against HBM bandwidth, otherwise against the matrix cores."""
    # fp32 4096^3: 682.7 FLOP/B, far above the fp32 ridge (19.7)
    fl, by = 2.0 * 4096 ** 3, 3 * 4096 * 4096 * 4
    r = bench.roofline_of(fl, by, 1.0, bench.PEAK["f32"], None)
    assert r["bound"] == "mfma" and r["unit"] == "TFLOP/s"
    assert abs(r["achieved"] - fl / 1e-3 / 1e12) < 0.01 and abs(r["frac"] - r["achieved"] / 157.3) < 1e-4
    # bf16-input conv 32x64x56x56 -> 64, 3x3: bf16 X and W, fp32 Y, 191.6 FLOP/B < 314.6
    fl = 2.0 * 32 * 64 * 56 * 56 * 64 * 9
    by = 32 * 64 * 56 * 56 * 2 + 64 * 64 * 9 * 2 + 32 * 64 * 56 * 56 * 4
    r = bench.roofline_of(fl, by, 0.02, bench.PEAK["bf16"], None)
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["achieved"] - by / 0.02e-3 / 1e9) < 0.1
    assert abs(r["ridge"] - 314.6) < 0.1 and r["intensity"] < r["ridge"]
