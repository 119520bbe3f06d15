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


def topp_accept(g: int, k: int, csum: np.ndarray, p: float) -> bool:
    """GPU cutoff g against the oracle's k on one row.  csum is the float64
    inclusive prefix of the row (non-negative entries, so it is also the
    prefix of |x|).  g is accepted if it equals k, or if the fp64 prefix at g
    is within tolerance of reaching p and the one before is within tolerance
    of not reaching it (tol_i = 1e-5 * csum_i + 1e-6)."""
    if g == k:
        return True
    n = csum.size
    if not (0 <= g < n):
        return False
    tol = FLOAT_REL * csum + FLOAT_ABS
    pd = float(np.float32(p))
    if g == n - 1 and csum[g] < pd + tol[g] and (g == 0 or csum[g - 1] < pd + tol[g - 1]):
        return True  # never reached within tolerance
    ok_here = csum[g] >= pd - tol[g]
    ok_before = g == 0 or csum[g - 1] < pd + tol[g - 1]
    return bool(ok_here and ok_before)


def draw_tol(theta: float, total: float) -> float:
    """Tolerance of a GPU threshold u = theta * total, where total is an fp32
    sum carrying the float bound and the product is rounded to fp32."""
    return theta * (FLOAT_REL * total + FLOAT_ABS) + 2.0**-23 * theta * total


def draw_accept(g: int, csum: np.ndarray, u: float, u_tol: float, limit: int) -> bool:
    """GPU inverse-transform draw g on one row: the first i <= limit whose
    running sum exceeds u, else limit.  csum is the float64 inclusive prefix
    of the row (non-negative entries); u the float64 threshold, known to the
    GPU within u_tol.  g is accepted if it lies in [0, limit], the prefix
    before it does not exceed u within tolerance, and its own prefix exceeds
    u within tolerance (or g is the fallback, limit)."""
    if not (0 <= g <= limit):
        return False
    tol = FLOAT_REL * csum + FLOAT_ABS + u_tol
    ok_here = csum[g] > u - tol[g]
    ok_before = g == 0 or csum[g - 1] <= u + tol[g - 1]
    return bool(ok_before and (ok_here or g == limit))
