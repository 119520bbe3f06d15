"""scan_inclusive_i32_noalloc (the entry point that allocates nothing: its
workspace is the library's static per-GPU array) against scan_inclusive_i32
(the same scan with a caller workspace) and the oracle, through the C ABI:
two calls in a row, the second on a smaller input, then an in-place call and
the size limit."""
import ctypes

import numpy as np
import pytest

import oracle
from gpu_util import announce, assert_equal_first_diff, to_dev, to_host
from paper_2505_15112_amd import _lib
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu

P = ctypes.c_void_p


def _ptr(t):
    return P(t.data_ptr())


def _both(lib, torch, x, stream):
    """(no-alloc result, workspace-entry-point result) for host array x."""
    n = x.size
    xd = to_dev(x)
    y0 = torch.empty_like(xd)
    y1 = torch.empty_like(xd)
    announce("scan_inclusive_i32_noalloc", n)
    assert lib.scan_inclusive_i32_noalloc(_ptr(xd), _ptr(y0), n, stream) == _lib.OK
    nbytes = _lib.workspace_bytes(_lib.OP_SCAN, n)
    ws = torch.zeros((nbytes + 15) // 16 * 16, dtype=torch.uint8, device=xd.device)
    announce("scan_inclusive_i32", n)
    assert lib.scan_inclusive_i32(_ptr(xd), _ptr(y1), n, _ptr(ws), ws.numel(), stream) == _lib.OK
    torch.cuda.synchronize()
    return to_host(y0), to_host(y1)


def test_noalloc_matches_workspace_entry_point_twice():
    import torch
    lib = _lib.load()
    stream = P(torch.cuda.current_stream().cuda_stream)
    # first call: the register + LDS tiles with a ragged last tile; second
    # call: smaller, other tile geometry, so stale status words of the first
    # call are in the array when it runs
    for n, seed in ((1 << 27) + 4099, 11), (300001, 12):
        x = W.scan_i32_full_range(n, seed=seed)
        got, want = _both(lib, torch, x, stream)
        assert_equal_first_diff(got, want, f"noalloc vs scan_inclusive_i32 n={n}")
        assert_equal_first_diff(got, oracle.scan_i32(x), f"noalloc vs oracle n={n}")


def test_noalloc_in_place_small_and_limits():
    import torch
    lib = _lib.load()
    stream = P(torch.cuda.current_stream().cuda_stream)
    for n in (1, 63, 4097, 70001):
        x = W.scan_i32(n, seed=n)
        xd = to_dev(x)
        announce("scan_inclusive_i32_noalloc in place", n)
        assert lib.scan_inclusive_i32_noalloc(_ptr(xd), _ptr(xd), n, stream) == _lib.OK
        torch.cuda.synchronize()
        assert_equal_first_diff(to_host(xd), oracle.scan_i32(x), f"in place n={n}")
    xd = torch.zeros(16, dtype=torch.int32, device="cuda")
    assert lib.scan_inclusive_i32_noalloc(_ptr(xd), _ptr(xd), 0, stream) == _lib.OK
    assert lib.scan_inclusive_i32_noalloc(_ptr(xd), _ptr(xd), -1, stream) == _lib.EINVAL
    # beyond the static workspace: rejected before any launch (the pointers
    # are never dereferenced)
    assert lib.scan_inclusive_i32_noalloc(P(1 << 40), P(1 << 42), (1 << 31) + 1,
                                          stream) == _lib.ERANGE
