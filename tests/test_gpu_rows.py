"""GPU parity of the batched row scans and the top-p cutoff (through the C ABI).

Row scans: int32 bit-exact, fp32 within the float bound plus bit-exact runs
on {-1, 0, 1}.  Shapes cover the one-wave-per-row schedule (len <= 1024), the
one-workgroup-per-row schedule (1024 < len <= 4096), the segmented look-back
schedule (len > 4096), ragged and unaligned lengths.
Top-p: the cutoff equals the oracle's, or lies inside the tolerance band
around p; dyadic rows (exact sums) must match exactly.
"""
import numpy as np
import pytest

import oracle
from gpu_util import (announce, assert_equal_first_diff, assert_float_close, to_dev, to_host,
                      topp_accept)
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu

SHAPES = [(1, 1), (3, 5), (7, 64), (5, 255), (6, 1024), (6, 1025), (33, 3001), (128, 4096),
          (4, 4096), (3, 4097), (2, 3 * 4096 + 5),
          (1000, 100), (17, 10_001), (9, 65_536), (3, 200_003)]


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("excl", [False, True])
def test_rows_i32(ops, shape, excl):
    rows, length = shape
    announce("rows i32", shape, excl)
    x = W.scan_i32_full_range(rows * length, seed=rows + length).reshape(rows, length)
    y = to_host(ops.scan_rows_i32(to_dev(x), exclusive=excl))
    assert_equal_first_diff(y, oracle.scan_rows_i32(x, exclusive=excl), f"rows i32 {shape}")


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("excl", [False, True])
def test_rows_f32(ops, shape, excl):
    rows, length = shape
    announce("rows f32", shape, excl)
    x = W.scan_f32(rows * length, seed=rows * length).reshape(rows, length)
    y = to_host(ops.scan_rows_f32(to_dev(x), exclusive=excl))
    ref, a = oracle.scan_rows_f32(x, exclusive=excl)
    assert_float_close(y.reshape(-1), ref.reshape(-1), a.reshape(-1), f"rows f32 {shape}")
    xe = W.exact_pm1(rows * length, seed=7).reshape(rows, length)
    ye = to_host(ops.scan_rows_f32(to_dev(xe), exclusive=excl))
    assert_equal_first_diff(ye.astype(np.float64), oracle.scan_rows_f32(xe, exclusive=excl)[0],
                            f"rows f32 exact {shape}")


def test_rows_inplace_and_empty(ops):
    import torch
    announce("rows in-place/empty")
    x = W.scan_i32_full_range(6 * 5000, seed=1).reshape(6, 5000)
    z = to_dev(x)
    ops.scan_rows_i32(z, out=z)
    assert_equal_first_diff(to_host(z), oracle.scan_rows_i32(x), "rows in-place")
    x2 = W.scan_i32_full_range(9 * 3000, seed=2).reshape(9, 3000)  # one workgroup per row
    z2 = to_dev(x2)
    ops.scan_rows_i32(z2, out=z2, exclusive=True)
    assert_equal_first_diff(to_host(z2), oracle.scan_rows_i32(x2, exclusive=True),
                            "rows in-place, one tile")
    assert ops.scan_rows_f32(torch.empty((0, 7), dtype=torch.float32, device="cuda")).numel() == 0
    assert ops.scan_rows_f32(torch.empty((7, 0), dtype=torch.float32, device="cuda")).numel() == 0


def _check_topp(ops, probs, p, what):
    g = to_host(ops.topp_cutoff_f32(to_dev(probs), p))
    k = oracle.topp_cutoff_f32(probs, p)
    csum, _ = oracle.scan_rows_f32(probs)
    bad = [r for r in range(probs.shape[0]) if not topp_accept(int(g[r]), int(k[r]), csum[r], p)]
    assert not bad, f"{what}: rows {bad[:5]} gpu {g[bad[:5]]} oracle {k[bad[:5]]}"
    return g, k


@pytest.mark.parametrize("length", [1, 3, 64, 255, 1000, 4096, 4097, 10_003, 3 * 4096 + 5,
                                    131_072])
@pytest.mark.parametrize("p", [0.0, 0.5, 0.9, 0.999, 1.5])
def test_topp_shapes(ops, length, p):
    announce("topp", length, p)
    probs = W.topp_probs(6, length, seed=length)
    _check_topp(ops, probs, p, f"topp len={length} p={p}")


@pytest.mark.parametrize("length", [64 * 32768, 64 * 32768 + 1, 65 * 32768 + 7])
@pytest.mark.parametrize("p", [0.5, 0.9, 1.5])
def test_topp_one_pass_limit(ops, length, p):
    """Rows of exactly 64 tiles (the last one-pass shape) and longer rows (the
    two-phase schedule)."""
    announce("topp long rows", length, p)
    probs = W.topp_probs(2, length, seed=length % 1000)
    _check_topp(ops, probs, p, f"topp len={length} p={p}")


@pytest.mark.parametrize("length", [8_191, 65_537, 131_072 + 5, 200_003, 262_145, 1 << 20,
                                    (1 << 20) + 1])
@pytest.mark.parametrize("p", [0.0, 0.5, 0.9, 0.999, 1.5])
def test_topp_early_exit_shapes(ops, length, p):
    """Rows of 2 to 256 tiles of 4096 take the early-exit kernel (2^20 + 1:
    the two-phase one); p = 1.5 reads every tile of every row, p = 0 stops in
    the first."""
    announce("topp early", length, p)
    probs = W.topp_probs(5, length, seed=length % 997)
    _check_topp(ops, probs, p, f"topp early len={length} p={p}")


@pytest.mark.parametrize("p", [0.3, 0.9])
def test_topp_early_exit_unsorted(ops, p):
    """The cutoff is defined on any row: unsorted softmax rows put the
    crossing in any tile."""
    announce("topp early unsorted", p)
    probs = W.sample_probs(7, 6 * 32768 + 11, seed=3)
    _check_topp(ops, probs, p, f"topp early unsorted p={p}")


@pytest.mark.parametrize("length", [12_289, 300_001])
def test_topp_early_exit_signed_walk(ops, length):
    """Rows of -1/0/+1 steps: the running sum crosses p, falls back and crosses
    again, so several tiles hold indices whose running sum reaches p and the
    cutoff is the first of them.  Every partial sum is a small integer, exact
    in fp32, so the GPU must match the oracle exactly."""
    announce("topp early signed walk", length)
    x = W.exact_pm1(6 * length, seed=length).reshape(6, length)
    walk = np.cumsum(x.astype(np.int64), axis=1)
    for p in (1.0, 3.0, float(max(1, walk.max() // 2)), 1e9):
        g = to_host(ops.topp_cutoff_f32(to_dev(x), p))
        k = oracle.topp_cutoff_f32(x, p)
        assert_equal_first_diff(g, k, f"signed walk len={length} p={p}")


def test_topp_early_exit_repeat(ops):
    """The early-exit kernels 30 times on one workspace, alternating p so that
    rows stop in different tiles (and p = 1.5 walks whole rows)."""
    from paper_2505_15112_amd import _lib
    import torch
    announce("topp early repeat")
    probs = W.topp_probs(64, 5 * 32768, seed=77)
    pd = to_dev(probs)
    ws = ops.workspace(_lib.OP_SCAN_ROWS, torch.device("cuda", 0), rows=64, length=5 * 32768)
    csum, _ = oracle.scan_rows_f32(probs)
    for it in range(30):
        p = (0.5, 0.9, 0.9999, 1.5)[it % 4]
        g = to_host(ops.topp_cutoff_f32(pd, p, ws=ws))
        k = oracle.topp_cutoff_f32(probs, p)
        bad = [r for r in range(64) if not topp_accept(int(g[r]), int(k[r]), csum[r], p)]
        assert not bad, (it, p, bad[:5])
    assert ops.workspace_error(ws) == 0


def test_topp_misaligned_view(ops):
    announce("topp misaligned")
    probs = W.topp_probs(3, 131_072 + 1, seed=5)
    d = to_dev(probs.reshape(-1))[1:1 + 3 * 131_072].reshape(3, 131_072)
    g = to_host(ops.topp_cutoff_f32(d, 0.9))
    host = probs.reshape(-1)[1:1 + 3 * 131_072].reshape(3, 131_072)
    k = oracle.topp_cutoff_f32(host, 0.9)
    csum, _ = oracle.scan_rows_f32(host)
    assert all(topp_accept(int(g[r]), int(k[r]), csum[r], 0.9) for r in range(3)), (g, k)


@pytest.mark.parametrize("m", [2, 7, 12, 13, 17, 18])
def test_topp_dyadic_exact(ops, m):
    """2^m equal probabilities 2^-m: every fp32 running sum is exact."""
    announce("topp dyadic", m)
    probs = np.full((3, 1 << m), 2.0**-m, np.float32)
    for p, want in ((0.5, (1 << (m - 1)) - 1), (1.0, (1 << m) - 1), (0.25, (1 << (m - 2)) - 1)):
        g = to_host(ops.topp_cutoff_f32(to_dev(probs), p))
        assert g.tolist() == [want] * 3, (m, p, g)


def test_topp_empty_rows(ops):
    import torch
    announce("topp empty")
    g = ops.topp_cutoff_f32(torch.empty((4, 0), dtype=torch.float32, device="cuda"), 0.9)
    assert to_host(g).tolist() == [-1] * 4


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_topp_config_128x131072(ops, seed):
    announce("topp config", seed)
    probs = W.topp_probs(128, 131_072, seed=seed)
    g, k = _check_topp(ops, probs, 0.9, f"topp config seed={seed}")
    # the cutoff sits near a quarter of the row for softmax(N(0, 4)) at p = 0.9
    assert 0.15 < float(np.median(k)) / 131_072 < 0.35


def test_rows_config_128x131072(ops):
    announce("rows config f32")
    probs = W.topp_probs(128, 131_072, seed=0)
    y = to_host(ops.scan_rows_f32(to_dev(probs)))
    ref, a = oracle.scan_rows_f32(probs)
    assert_float_close(y.reshape(-1), ref.reshape(-1), a.reshape(-1), "rows config")
