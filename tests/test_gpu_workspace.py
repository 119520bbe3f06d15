"""The workspace contract on the GPU: zero-filled once, then shared by any
sequence of calls of any op, never cleared again -- including across the
once-in-2^30-calls wrap of the 30-bit status epoch, which is forced here by
writing the header's epoch from the host.  A header that was never
initialised must make the kernel raise the error word and finish (no hang).
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, assert_equal_first_diff, assert_float_close, to_dev, to_host
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


def _big_ws(ops, n):
    import torch
    from paper_2505_15112_amd import _lib
    sizes = [_lib.workspace_bytes(_lib.OP_SCAN, n), _lib.workspace_bytes(_lib.OP_SCAN_RSS, n),
             _lib.workspace_bytes(_lib.OP_COMPACT, n),
             _lib.workspace_bytes(_lib.OP_RADIX_SORT, n, bits=8),
             _lib.workspace_bytes(_lib.OP_RADIX_SORT, n, bits=4),
             _lib.workspace_bytes(_lib.OP_RADIX_SORT, n, bits=1),
             _lib.workspace_bytes(_lib.OP_SCAN_ROWS, rows=16, length=n // 16),
             _lib.workspace_bytes(_lib.OP_SORT_ROWS, rows=16, length=n // 16),
             _lib.workspace_bytes(_lib.OP_WEIGHTED_SAMPLE, rows=16, length=n // 16),
             _lib.workspace_bytes(_lib.OP_TOPP_SAMPLE, rows=16, length=n // 16)]
    nbytes = (max(sizes) + 15) // 16 * 16
    return torch.zeros(nbytes, dtype=torch.uint8, device="cuda")  # zero-filled = ready


def _run_all(ops, ws, n, seed):
    """Every op on one workspace, each checked against the oracle."""
    x = W.scan_i32_full_range(n, seed=seed)
    xd = to_dev(x)
    assert_equal_first_diff(to_host(ops.scan_inclusive_i32(xd, ws=ws)), oracle.scan_i32(x), "scan")
    assert_equal_first_diff(to_host(ops.scan_inclusive_rss_i32(xd, ws=ws)), oracle.scan_i32(x), "rss")
    xf = W.scan_f32(n, seed=seed)
    ref, a = oracle.scan_f32(xf, exclusive=True)
    assert_float_close(to_host(ops.scan_exclusive_f32(to_dev(xf), ws=ws)), ref, a, "scan f32")
    m = W.mask_u8(n, seed=seed)
    out, idx, cnt = ops.compact_by_mask_f32(to_dev(xf), to_dev(m), with_idx=True, ws=ws)
    ro, ri = oracle.compact_f32(xf, m)
    assert int(cnt.item()) == ro.size
    assert_equal_first_diff(to_host(idx)[: ro.size], ri, "compact idx")
    k = W.keys_u32(n, seed=seed)
    ko, io, nt = ops.split_by_flags_u32(to_dev(k.view(np.int32)), to_dev(m), ws=ws)
    rk, rio, rn = oracle.split_u32(k, m)
    assert int(nt.item()) == rn
    assert_equal_first_diff(to_host(io), rio, "split idx")
    rk, rp = oracle.sort_u32(k)
    for bits in (8, 4, 1):
        so, sp = ops.radix_sort_u32(to_dev(k.view(np.int32)), bits_per_pass=bits, ws=ws)
        assert_equal_first_diff(to_host(sp), rp, f"radix{bits}")
    xr = x.reshape(16, n // 16)
    assert_equal_first_diff(to_host(ops.scan_rows_i32(to_dev(xr), ws=ws)), oracle.scan_rows_i32(xr),
                            "rows")
    _check_topp(ops, ws, n, seed)
    _check_samplers(ops, ws, n, seed)


def _check_samplers(ops, ws, n, seed):
    """The row sort and both samplers, exact cases (integer-valued sums): the
    sort's count table and the samplers' tile sums share the workspace with
    everything above."""
    rng = np.random.default_rng(seed)
    k = W.values_f32(n, seed=seed).reshape(16, n // 16)
    ko, po = ops.radix_sort_rows_f32(to_dev(k), descending=True, ws=ws)
    rk, rp = oracle.sort_rows_f32(k, descending=True)
    assert_equal_first_diff(to_host(po), rp, "sort rows")
    w = rng.integers(0, 4, (16, n // 16)).astype(np.float32)
    theta = (rng.integers(0, 4, 16) / 4.0).astype(np.float32)
    g = to_host(ops.weighted_sample_f32(to_dev(w), to_dev(theta), ws=ws))
    assert_equal_first_diff(g, oracle.weighted_sample_f32(w, theta), "weighted")
    probs = (rng.integers(0, 16, (16, n // 16)) * 2.0**-24).astype(np.float32)
    tok = to_host(ops.topp_sample_f32(to_dev(probs), to_dev(theta), 2.0**-6, ws=ws))
    assert_equal_first_diff(tok, oracle.topp_sample_f32(probs, theta, 2.0**-6)[0], "topp sample")


def _check_topp(ops, ws, n, seed):
    from gpu_util import topp_accept
    # 16 rows of n/16 and 4 rows of 32 tiles of 4096 (the early-exit
    # kernels, whose head words share the workspace too)
    for shape in ((16, n // 16), (4, 4 * 32768 + 5)):
        probs = W.topp_probs(shape[0], shape[1], seed=seed)
        g = to_host(ops.topp_cutoff_f32(to_dev(probs), 0.9, ws=ws))
        k = oracle.topp_cutoff_f32(probs, 0.9)
        csum, _ = oracle.scan_rows_f32(probs)
        bad = [r for r in range(shape[0]) if not topp_accept(int(g[r]), int(k[r]), csum[r], 0.9)]
        assert not bad, ("topp", shape, bad, g[bad], k[bad])


def test_one_workspace_for_every_op(ops):
    announce("shared workspace, all ops")
    n = 16 * 40_000
    ws = _big_ws(ops, n)
    ops.set_checked(True)  # every op's call is followed by a read of the error word
    try:
        for seed in range(3):
            _run_all(ops, ws, n, seed)
    finally:
        ops.set_checked(False)
    assert ops.workspace_error(ws) == 0


def test_epoch_wrap(ops):
    """Set the header epoch to the last value before the 30-bit status tag
    wraps: that call must clear the workspace, and every later call of every
    op must still be right."""
    import torch
    announce("epoch wrap")
    n = 16 * 40_000
    ws = _big_ws(ops, n)
    _run_all(ops, ws, n, 7)  # leaves live-looking status words of low epochs
    hdr = ws[:8].view(torch.int64)
    hdr.copy_(torch.tensor([((1 << 30) - 1) << 32], dtype=torch.int64, device=ws.device))
    torch.cuda.synchronize()
    x = W.scan_i32_full_range(n, seed=8)
    assert_equal_first_diff(to_host(ops.scan_inclusive_i32(to_dev(x), ws=ws)), oracle.scan_i32(x),
                            "wrap call")
    epoch = int(ws[:8].view(torch.int64).cpu()[0]) >> 32
    assert epoch == 1 << 30
    for seed in (9, 10):
        _run_all(ops, ws, n, seed)
    assert ops.workspace_error(ws) == 0


def test_topp_after_row_scan_at_high_epoch(ops):
    """A row scan at an epoch >= 2^29 leaves status words whose bit 61 is set
    where top-p keeps its tile sums; top-p on the same workspace must not take
    them for sums."""
    import torch
    announce("topp after high-epoch row scan")
    n = 16 * 40_000
    ws = _big_ws(ops, n)
    ws[:8].view(torch.int64).copy_(torch.tensor([((1 << 29) + 5) << 32], dtype=torch.int64,
                                                device=ws.device))
    for seed in (11, 12):
        x = W.scan_i32_full_range(n, seed=seed).reshape(16, n // 16)
        assert_equal_first_diff(to_host(ops.scan_rows_i32(to_dev(x), ws=ws)),
                                oracle.scan_rows_i32(x), "rows at high epoch")
        _check_topp(ops, ws, n, seed)
    assert ops.workspace_error(ws) == 0


def test_uninitialised_header_raises_error_word(ops):
    """Tickets that start past the grid: the workgroup sets the error word and
    finishes instead of waiting for tiles nobody will process."""
    import torch
    from paper_2505_15112_amd import _lib
    announce("uninitialised header")
    n = 1000  # one tile
    ws = ops.workspace(_lib.OP_SCAN, torch.device("cuda", 0), n)
    ws[:8].view(torch.int64).fill_(5)  # ticket count 5: the only workgroup draws ticket 5
    x = to_dev(W.scan_i32(n, seed=1))
    ops.scan_inclusive_i32(x, ws=ws)
    torch.cuda.synchronize()
    assert ops.workspace_error(ws, reset=False) == 1
    assert ops.workspace_error(ws) == 1  # read again, then cleared
    assert ops.workspace_error(ws) == 0
    ops.scan_inclusive_i32(x, ws=ws)  # the ticket count is still past the grid: set again
    assert ops.workspace_error(ws) == 1
    # checked mode: the binding reads the word after the call and raises
    ops.set_checked(True)
    try:
        with pytest.raises(_lib.LibscanError, match="error word"):
            ops.scan_inclusive_i32(x, ws=ws)
    finally:
        ops.set_checked(False)
