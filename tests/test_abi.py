"""C ABI of libxtc.so on the CPU: the library loads without a GPU, exports
every function include/xtc.h declares, and rejects every invalid call with the
documented status before touching the device (all checks below use NULL or
dummy pointers, which a kernel would fault on, so a wrong OK would show)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "xtc.h")


@pytest.fixture(scope="module")
def x():
    import paper_2512_16512_amd as mod
    return mod


def _declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(xtc_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_abi():
    names = _declared_functions()
    for n in ("xtc_matmul", "xtc_conv2d_nchw", "xtc_default_schedule", "xtc_sched_check",
              "xtc_sched_list", "xtc_status_str"):
        assert n in names


def test_library_exports_every_declared_symbol(x):
    lib = ctypes.CDLL(x.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), "libxtc.so does not export %s" % name
    assert sorted(x.EXPORTS) == _declared_functions()


def test_sched_struct_size_matches_header(x):
    src = open(HEADER).read()
    body = re.search(r"typedef struct \{(.*?)\} xtc_sched;", src, re.S).group(1)
    n_fields = len(re.findall(r"\b[a-z_]+\b(?=[,;])", re.sub(r"/\*.*?\*/", "", body, flags=re.S)))
    assert ctypes.sizeof(x.Sched) == 4 * n_fields


def test_status_strings(x):
    for st in range(0, 10):
        s = x.xtc_status_str(st)
        assert s and s != "unknown status"
    assert x.xtc_status_str(99) == "unknown status"


BAD = 0x10  # a dummy non-NULL pointer: dereferencing it would fault


@pytest.mark.parametrize("args,expected", [
    ((-1, 4, 4, BAD, 4, BAD, 4, BAD, 4, 0), 2),          # negative M
    ((4, -1, 4, BAD, 4, BAD, 4, BAD, 4, 0), 2),          # negative N
    ((4, 4, -1, BAD, 4, BAD, 4, BAD, 4, 0), 2),          # negative K
    ((4, 4, 8, BAD, 7, BAD, 4, BAD, 4, 0), 3),           # lda < K
    ((4, 8, 4, BAD, 4, BAD, 7, BAD, 8, 0), 3),           # ldb < N
    ((4, 8, 4, BAD, 4, BAD, 8, BAD, 7, 0), 3),           # ldc < N
    ((4, 4, 4, BAD, 4, BAD, 4, BAD, 4, 7), 4),           # unknown dtype
    ((4, 4, 4, 0, 4, BAD, 4, BAD, 4, 0), 1),             # A NULL
    ((4, 4, 4, BAD, 4, 0, 4, BAD, 4, 0), 1),             # B NULL
    ((4, 4, 4, BAD, 4, BAD, 4, 0, 4, 0), 1),             # C NULL
    ((1 << 16, 1 << 15, 1 << 15, BAD, 1 << 15, BAD, 1 << 15, BAD, 1 << 15, 0), 7),  # span >= 2^31
    ((3, 3, 1 << 30, BAD, 1 << 30, BAD, 3, BAD, 3, 1), 7),
    ((1, 1, 0x1FFFFFF5, BAD, 0x1FFFFFF5, BAD, 1, BAD, 1, 0), 7),  # span 0x7FFFFFD4 > 0x7FFFFFD0
    # (M - 1) * ld = 2^64 would wrap to 0 and leave spans of 16 bytes
    (((1 << 62) + 1, 4, 4, BAD, 4, BAD, 4, BAD, 4, 0), 7),
    ((2**63 - 1, 2**63 - 1, 2**63 - 1, BAD, 2**63 - 1, BAD, 2**63 - 1, BAD, 2**63 - 1, 1), 7),
    ((4, 4, 4, BAD + 2, 4, BAD, 4, BAD, 4, 0), 9),       # fp32 A on a 2-byte boundary
    ((4, 4, 4, BAD, 4, BAD + 1, 4, BAD, 4, 1), 9),       # bf16 B on an odd byte
    ((4, 4, 4, BAD, 4, BAD, 4, BAD + 2, 4, 1), 9),       # C (fp32) on a 2-byte boundary
])
def test_matmul_validation(x, args, expected):
    assert x.xtc_matmul(*args) == expected
    assert x.xtc_matmul_relu(*args) == expected


def test_matmul_empty_is_noop(x):
    # M == 0 or N == 0 returns OK without any device work (NULL pointers allowed)
    assert x.xtc_matmul(0, 5, 5, 0, 5, 0, 5, 0, 5, 0) == 0
    assert x.xtc_matmul(5, 0, 5, 0, 5, 0, 1, 0, 1, 1) == 0
    assert x.xtc_matmul_relu(0, 5, 5, 0, 5, 0, 5, 0, 5, 0) == 0


@pytest.mark.parametrize("args,expected", [
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, 0, BAD, BAD, 1), 1),       # bf16 conv, X NULL
    ((1, 1024, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD, BAD, 1), 7),  # bf16: C*R*S > table capacity
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD, BAD, 5), 4),     # unknown dtype
    ((1, 0, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD, BAD, 0), 2),     # C = 0
    ((1, 3, 8, 8, 4, 3, 3, 0, 1, 1, 1, BAD, BAD, BAD, 0), 2),     # stride 0
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, -1, 1, BAD, BAD, BAD, 0), 2),    # negative pad
    ((1, 3, 2, 2, 4, 5, 5, 1, 1, 0, 0, BAD, BAD, BAD, 0), 2),     # kernel larger than input
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, 0, BAD, BAD, 0), 1),       # X NULL
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, 0, BAD, 0), 1),       # W NULL
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD, 0, 0), 1),       # Y NULL
    ((1, 1024, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD, BAD, 0), 7),  # C*R*S > table capacity
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD + 2, BAD, BAD, 0), 9),  # fp32 X on a 2-byte boundary
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD + 1, BAD, 1), 9),  # bf16 W on an odd byte
    ((1, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, BAD, BAD, BAD + 2, 1), 9),  # Y on a 2-byte boundary
    # strides, pads and padded extents above 2^30 (coordinates must stay in
    # 32-bit arithmetic): a stride of 2^34 and a pad of 2^32 on a 3x3 input
    # would give OH = 1 and pass every other check
    ((1, 1, 3, 3, 1, 3, 3, 1 << 34, 1, 1 << 32, 0, BAD, BAD, BAD, 0), 7),
    ((1, 1, 3, 3, 1, 3, 3, 1, 1 << 31, 0, 0, BAD, BAD, BAD, 0), 7),
    ((1, 1, 3, 3, 1, 3, 3, 1, 1, 0, (1 << 30) + 1, BAD, BAD, BAD, 0), 7),
    ((1, 1, 3, 3, 1, 3, 3, 1, 1, 1 << 29, 0, BAD, BAD, BAD, 0), 7),   # H + 2*pad_h > 2^30
    # X and Y spans of 2^61 x 16 x 4 bytes would wrap to 0
    ((1 << 61, 1, 4, 4, 1, 3, 3, 1, 1, 0, 0, BAD, BAD, BAD, 0), 7),
    ((1, 1 << 62, 4, 4, 1, 3, 3, 1, 1, 0, 0, BAD, BAD, BAD, 0), 7),   # C * R * S wraps
    ((2**63 - 1, 2**63 - 1, 3, 3, 2**63 - 1, 3, 3, 1, 1, 0, 0, BAD, BAD, BAD, 1), 7),
])
def test_conv_validation(x, args, expected):
    assert x.xtc_conv2d_nchw(*args) == expected
    assert x.xtc_conv2d_nchw_relu(*args) == expected


def test_conv_empty_is_noop(x):
    assert x.xtc_conv2d_nchw(0, 3, 8, 8, 4, 3, 3, 1, 1, 1, 1, 0, 0, 0, 0) == 0
    assert x.xtc_conv2d_nchw(2, 3, 8, 8, 0, 3, 3, 1, 1, 1, 1, 0, 0, 0, 0) == 0


def test_sched_list_and_check(x):
    for op, dt in ((0, 0), (0, 1), (1, 0), (1, 1)):
        lst = x.xtc_sched_list(op, dt)
        assert len(lst) >= 3
        for s in lst:
            assert x.xtc_sched_check(op, dt, s) == 0
            for r in (0, 1, 4, 8):           # raster and xcd remap are run-time choices
                s2 = x.Sched(**s.as_dict())
                s2.raster = r
                s2.xcd_remap = r & 1
                assert x.xtc_sched_check(op, dt, s2) == 0
    assert x.xtc_sched_list(1, 2) == [] and x.xtc_sched_list(2, 0) == []


def _base(x, dt=0):
    return x.Sched(**x.xtc_sched_list(0, dt)[0].as_dict())


@pytest.mark.parametrize("field,value", [
    ("block_m", 96), ("block_n", 0), ("wave_m", 512), ("mfma_m", 8), ("mfma_k", 16),
    ("lds_stages", 0), ("lds_pad", -2), ("raster", -1), ("xcd_remap", 2), ("block_k", 4),
    ("raster", 65), ("raster", 1 << 28), ("raster", 2**31 - 1),
    ("size", 12), ("k_order", 1), ("k_order", -1), ("k_split", 0), ("k_split", 3),
    ("k_split", 16),
])
def test_sched_illegal_fields(x, field, value):
    s = _base(x)
    setattr(s, field, value)
    assert x.xtc_sched_check(0, 0, s) == 5
    # and the same schedule is refused by the entry point before any device work
    assert x.xtc_matmul(4, 4, 4, BAD, 4, BAD, 4, BAD, 4, 0, s) == 5
    assert x.xtc_matmul_relu(4, 4, 4, BAD, 4, BAD, 4, BAD, 4, 0, s) == 5


def test_sched_legal_but_not_compiled(x):
    s = _base(x)
    s.block_m, s.block_n, s.wave_m, s.wave_n = 64, 128, 32, 64
    assert x.xtc_sched_check(0, 0, s) == 6
    assert x.xtc_matmul(4, 4, 4, BAD, 4, BAD, 4, BAD, 4, 0, s) == 6


def test_sched_non_power_of_two_pixel_tiles(x):
    # A pixel tile that is not a power of two (208 = 13 instruction blocks of
    # 16) is legal only for the conv kernels that stage an input patch
    # (k_order 2), whose block_k counts channels per stage; the compiled
    # balanced halo instance is one such schedule.
    conv = [s for s in x.xtc_sched_list(x.XTC_OP_CONV2D, x.XTC_F32) if s.block_n == 208]
    assert len(conv) == 1 and conv[0].k_order == 2 and conv[0].block_k == 8
    assert x.xtc_sched_check(x.XTC_OP_CONV2D, x.XTC_F32, conv[0]) == 0
    s = x.Sched(**conv[0].as_dict())
    s.k_order = 1                       # other reduction orders: powers of two only
    assert x.xtc_sched_check(x.XTC_OP_CONV2D, x.XTC_F32, s) == 5
    s = x.Sched(**conv[0].as_dict())
    s.block_n = s.wave_n = 200          # not a whole number of 16-pixel blocks
    assert x.xtc_sched_check(x.XTC_OP_CONV2D, x.XTC_F32, s) == 5
    s = x.Sched(**conv[0].as_dict())
    s.block_n = s.wave_n = 224          # legal, but not compiled
    assert x.xtc_sched_check(x.XTC_OP_CONV2D, x.XTC_F32, s) == 6
    m = _base(x)
    m.block_n, m.wave_n = 208, 208      # never for matmul
    assert x.xtc_sched_check(x.XTC_OP_MATMUL, x.XTC_F32, m) == 5


def test_sched_lds_budget(x):
    s = _base(x, 1)
    s.block_m = s.block_n = 512
    s.wave_m, s.wave_n = 128, 128
    assert x.xtc_sched_check(0, 1, s) == 5


def test_bf16_schedule_rejected_for_f32(x):
    s = _base(x, 1)
    assert x.xtc_sched_check(0, 0, s) == 5


def test_default_schedules_are_compiled(x):
    for (op, dt, M, N, K) in [(0, 0, 4096, 4096, 4096), (0, 0, 256, 256, 256), (0, 0, 1, 1, 1),
                              (0, 1, 8192, 8192, 8192), (0, 1, 100, 100, 100), (0, 1, 2048, 2048, 64),
                              (1, 0, 64, 100352, 576), (1, 0, 256, 1000, 2304),
                              (1, 0, 16, 12544, 147), (1, 1, 64, 100352, 576), (1, 1, 16, 12544, 147),
                              (1, 1, 256, 1000, 2304)]:
        s = x.xtc_default_schedule(op, dt, M, N, K)
        assert x.xtc_sched_check(op, dt, s) == 0, (op, dt, M, N, K, s)
    with pytest.raises(x.XtcError):
        x.xtc_default_schedule(1, 2, 64, 64, 64)
    # extents up to 2^63 - 1 (tile counts saturate instead of wrapping)
    for op in (0, 1):
        for dt in (0, 1):
            for M, N in [(2**63 - 1, 2**63 - 1), (1, 2**63 - 1), (2**63 - 1, 1)]:
                s = x.xtc_default_schedule(op, dt, M, N, 2**63 - 1)
                assert x.xtc_sched_check(op, dt, s) == 0


def test_no_hip_error_recorded_by_validation(x):
    assert x.xtc_last_hip_error() == 0
    assert x.xtc_conv_max_k() >= 576


def test_one_hip_runtime_whatever_the_import_order():
    # The binding loads torch before libxtc.so, so the process maps a single
    # HIP runtime (two would make torch's device pointers invalid handles for
    # the library's launches).
    import subprocess
    import sys
    code = ("import paper_2512_16512_amd\nimport torch\n"
            "print(len({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, cwd=ROOT)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().splitlines()[-1] == "1"


def test_k_split_rules(x):
    # register-fed split: each wave covers the whole tile, nothing in LDS
    ks = [s for s in x.xtc_sched_list(0, 0) if s.k_split > 1 and s.lds_stages == 0]
    assert ks, "no reduction-split fp32 instance compiled"
    s = x.Sched(**ks[0].as_dict())
    assert x.xtc_sched_check(0, 0, s) == 0
    bad = x.Sched(**s.as_dict())
    bad.wave_m = s.block_m // 2            # register-fed split waves must cover the whole tile
    assert x.xtc_sched_check(0, 0, bad) == 5
    bad = x.Sched(**s.as_dict())
    bad.lds_stages = 2                     # legal (an LDS-staged split), not compiled for this tile
    assert x.xtc_sched_check(0, 0, bad) == 6
    # LDS-staged split: groups of waves, each running the staged pipeline on
    # its share of the K-steps
    st = [s for s in x.xtc_sched_list(0, 0) if s.k_split > 1 and s.lds_stages > 0]
    assert st and all(t.wave_m < t.block_m for t in st)
    assert x.xtc_sched_check(0, 0, st[0]) == 0
    bad = x.Sched(**st[0].as_dict())
    bad.lds_stages = 0                     # smaller waves than the tile need the LDS pipeline
    assert x.xtc_sched_check(0, 0, bad) == 5
    bad = x.Sched(**s.as_dict())
    bad.k_split = 2                        # legal value, not compiled
    assert x.xtc_sched_check(0, 0, bad) in (0, 6)
    conv = x.Sched(**x.xtc_sched_list(1, 0)[0].as_dict())
    conv.k_split = 2
    assert x.xtc_sched_check(1, 0, conv) == 5
    assert x.Sched().k_split == 1          # the Python default


def test_occupancy_query_validation(x):
    import ctypes
    s = x.xtc_sched_list(0, 0)[0]
    n = ctypes.c_int32(-1)
    lib = x._lib
    assert lib.xtc_sched_occupancy(0, 0, 64, None, ctypes.byref(n)) == 1
    assert lib.xtc_sched_occupancy(0, 0, 64, ctypes.byref(s), None) == 1
    assert lib.xtc_sched_occupancy(0, 0, -1, ctypes.byref(s), ctypes.byref(n)) == 2
    bad = x.Sched(**s.as_dict())
    bad.block_m = 96
    assert lib.xtc_sched_occupancy(0, 0, 64, ctypes.byref(bad), ctypes.byref(n)) == 5
    c = x.xtc_sched_list(1, 0)[0]
    assert lib.xtc_sched_occupancy(1, 0, 5000, ctypes.byref(c), ctypes.byref(n)) == 7
    assert n.value == -1                  # nothing written on an error
