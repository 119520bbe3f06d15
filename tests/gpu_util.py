"""Helpers shared by the GPU parity tests (host <-> device, tolerances)."""
import os
import sys

import numpy as np

FLOAT_REL = 1e-5   # |y_i - ref_i| <= FLOAT_REL * sum_{j<=i}|x_j| + FLOAT_ABS
FLOAT_ABS = 1e-6


def torch_dev():
    import torch
    return torch, torch.device("cuda", 0)


def to_dev(a: np.ndarray):
    torch, dev = torch_dev()
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def to_host(t) -> np.ndarray:
    return t.detach().cpu().numpy()


def announce(*parts):
    """Name the case on stdout (flushed) before each GPU step."""
    print("[gpu-case]", *parts, flush=True)
    sys.stdout.flush()


def assert_float_close(y: np.ndarray, ref: np.ndarray, absref: np.ndarray, what=""):
    """The float bound: |y_i - ref_i| <= 1e-5 * prefix(|x|)_i + 1e-6."""
    y = y.astype(np.float64)
    err = np.abs(y - ref)
    tol = FLOAT_REL * absref + FLOAT_ABS
    bad = ~(err <= tol)  # NaN counts as bad
    if bad.any():
        i = int(np.flatnonzero(bad)[0])
        raise AssertionError(f"{what}: {int(bad.sum())} elements out of tolerance; first at {i}: "
                             f"got {y[i]!r}, ref {ref[i]!r}, tol {tol[i]!r}")


def assert_equal_first_diff(got: np.ndarray, want: np.ndarray, what=""):
    if got.shape != want.shape:
        raise AssertionError(f"{what}: shape {got.shape} != {want.shape}")
    ne = got != want
    if ne.any():
        i = int(np.flatnonzero(ne.reshape(-1))[0])
        g, w = got.reshape(-1)[i], want.reshape(-1)[i]
        raise AssertionError(f"{what}: {int(ne.sum())} mismatches; first at {i}: got {g!r}, "
                             f"want {w!r}")


FULL = os.environ.get("LIBSCAN_FULL_SIZE_TESTS", "1") == "1"
