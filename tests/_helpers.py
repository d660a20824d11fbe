"""Shared helpers of the GPU tests: device transfer of the seeded inputs and
the parity assertion.  Inputs come from xtc_inputs only; expected values come
from the oracle only."""
import sys

import numpy as np

import oracle

TOL = {"f32": 1e-5, "bf16": 1e-2}


def say(*a):
    """Name the case before a GPU step (flushed, so a fault still shows it)."""
    print("[gpu]", *a, flush=True)
    sys.stdout.flush()


def to_dev(arr):
    """numpy fp32 array, or uint16 bf16-bit array, -> torch CUDA tensor."""
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).cuda()


def to_host(t):
    import torch
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def assert_parity(got, ref, dtype, what=""):
    err = oracle.rel_fro(got, ref)
    tol = TOL[dtype]
    assert np.all(np.isfinite(got)), "%s: non-finite output" % what
    assert err <= tol, "%s: rel Frobenius error %.3e > %.0e" % (what, err, tol)
    return err
