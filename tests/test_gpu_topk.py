"""GPU parity of top-k per row (through the C ABI) against the oracle.

Top-k's result is unique (the first k entries of the stable sort in the
asked direction, IEEE 754 totalOrder), so values are compared bit for bit
and indices exactly: ties (heavy, from small integers), signed zeros,
infinities and NaNs of both signs, k = 1, k = len, rows of one tile and of
many, ragged and misaligned rows, both directions.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, assert_equal_first_diff, to_dev, to_host
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


def _check(ops, x, k, largest, what):
    v, i = ops.topk_rows_f32(to_dev(x), k, largest=largest)
    rv, ri = oracle.topk_rows_f32(x, k, largest=largest)
    assert_equal_first_diff(to_host(i), ri, f"{what} indices")
    assert_equal_first_diff(to_host(v).view(np.uint32), rv.view(np.uint32), f"{what} values")


def _rows(rows, length, seed, kind):
    if kind == "normal":
        return W.values_f32(rows * length, seed=seed).reshape(rows, length)
    if kind == "ties":  # few distinct values: long runs of equal keys
        rng = np.random.default_rng(seed)
        return rng.integers(-3, 4, (rows, length)).astype(np.float32)
    if kind == "special":
        x = W.values_f32(rows * length, seed=seed).reshape(rows, length)
        rng = np.random.default_rng(seed + 1)
        sp = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, -np.nan, 1.0], np.float32)
        pick = rng.random((rows, length)) < 0.1
        x[pick] = sp[rng.integers(0, sp.size, int(pick.sum()))]
        return x
    if kind == "probs":
        return W.sample_probs(rows, length, seed=seed)
    raise ValueError(kind)


SHAPES = [(1, 1, [1]), (3, 5, [1, 2, 5]), (1000, 100, [1, 10, 100]), (4, 4096, [1, 64, 4096]),
          (3, 4097, [100, 4097]), (7, 10_001, [1, 1000]), (2, 3 * 8192 + 5, [5000]),
          (9, 65_536, [50, 4096]), (3, 65_537, [3]), (16, 131_072, [1, 4096]),
          (3, 200_003, [2000]), (4, 20_000, [8191, 8192, 8193]), (1, (1 << 20) + 3, [1, 70_000]),
          # the small-k route (k <= 256, rows up to 2^17): ragged last tiles
          # with fewer keys than k, its boundary at k = 256 / 257, and the
          # finisher's three LDS sizes
          (2, 3 * 8192 + 5, [7, 256]), (5, 16_385, [256, 257]), (3, 16_384, [200]),
          (2, 2048, [256]), (6, 131_072, [256, 257])]
# k <= 8192: the kept elements are ordered by an LDS sort per row; above, by the row radix sort


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("kind", ["normal", "ties", "special"])
@pytest.mark.parametrize("largest", [True, False])
def test_topk(ops, shape, kind, largest):
    rows, length, ks = shape
    for k in ks:
        announce("topk", rows, length, k, kind, largest)
        x = _rows(rows, length, seed=rows + length + k, kind=kind)
        _check(ops, x, k, largest, f"topk {rows}x{length} k={k} {kind} largest={largest}")


def test_topk_all_equal_and_k0(ops):
    import torch
    announce("topk all equal / k=0")
    x = np.full((5, 50_000), 0.25, np.float32)
    _check(ops, x, 7, True, "all equal")          # the first k indices
    _check(ops, x, 50_000, False, "all equal, k = len")
    v, i = ops.topk_rows_f32(torch.empty((3, 10), dtype=torch.float32, device="cuda"), 0)
    assert v.shape == (3, 0) and i.shape == (3, 0)


def test_topk_misaligned(ops):
    announce("topk misaligned")
    flat = _rows(1, 4 * 40_000 + 1, seed=11, kind="ties").reshape(-1)
    d = to_dev(flat)[1:].reshape(4, 40_000)  # 4-byte aligned, not 16-byte aligned
    assert d.data_ptr() % 16 != 0
    v, i = ops.topk_rows_f32(d, 333)
    rv, ri = oracle.topk_rows_f32(flat[1:].reshape(4, 40_000), 333)
    assert_equal_first_diff(to_host(i), ri, "misaligned indices")
    assert_equal_first_diff(to_host(v).view(np.uint32), rv.view(np.uint32), "misaligned values")


def test_topk_misaligned_small_k(ops):
    """The small-k route on misaligned rows (element-wise loads, twice the
    waves per tile)."""
    announce("topk misaligned small k")
    flat = _rows(1, 3 * 70_000 + 1, seed=12, kind="normal").reshape(-1)
    d = to_dev(flat)[1:].reshape(3, 70_000)
    assert d.data_ptr() % 16 != 0
    for k in (1, 50, 256):
        v, i = ops.topk_rows_f32(d, k)
        rv, ri = oracle.topk_rows_f32(flat[1:].reshape(3, 70_000), k)
        assert_equal_first_diff(to_host(i), ri, f"misaligned k={k} indices")
        assert_equal_first_diff(to_host(v).view(np.uint32), rv.view(np.uint32),
                                f"misaligned k={k} values")


@pytest.mark.parametrize("n_t", [1024, 1025])
@pytest.mark.parametrize("largest", [True, False])
def test_topk_tile_slot_edges(ops, n_t, largest):
    """On the small-k route every 8192-element tile keeps its keys whose top 16
    key bits are at least its own k-th key's, in 1024 slots; a tile with more
    sends its row the long way.  Here one tile of the middle row holds n_t
    values sharing their top 16 bits (2 + i * 2^-20), with ties among them,
    above (below, for the smallest k) the rest of the row, which is normal
    data of small magnitude."""
    announce("topk tile slots", n_t, largest)
    rows, length, k = 3, 131_072, 100
    rng = np.random.default_rng(n_t)
    x = (W.values_f32(rows * length, seed=n_t).reshape(rows, length) * 0.1).astype(np.float32)
    pos = 5 * 8192 + rng.choice(8192, n_t, replace=False)
    big = (2.0 + rng.integers(0, 64, n_t) * 2.0**-20).astype(np.float32)
    x[1, pos] = big if largest else -big
    _check(ops, x, k, largest, f"tile slots n_t={n_t} largest={largest}")


@pytest.mark.parametrize("k", [64, 4096])
def test_topk_config_128x131072(ops, k):
    announce("topk config", k)
    _check(ops, _rows(128, 131_072, seed=k, kind="probs"), k, True, f"config k={k}")


def test_topk_repeated_calls_share_workspace(ops):
    """Calls of different shapes on one workspace (status chains, digit counts,
    row states and counters left by one call must not disturb the next)."""
    import torch
    from paper_2505_15112_amd import _lib
    announce("topk shared workspace")
    dev = torch.device("cuda", 0)
    big = max(_lib.workspace_bytes(_lib.OP_TOPK, 4096, rows=64, length=131_072),
              _lib.workspace_bytes(_lib.OP_SCAN, 1 << 22),
              _lib.workspace_bytes(_lib.OP_RADIX_SORT, 1 << 22, bits=8))
    ws = torch.zeros((big + 15) // 16 * 16, dtype=torch.uint8, device=dev)
    for seed, (rows, length, k) in enumerate([(64, 131_072, 4096), (5, 70_001, 9),
                                              (64, 131_072, 4096), (300, 1000, 999)]):
        x = _rows(rows, length, seed=seed, kind="ties" if seed % 2 else "normal")
        v, i = ops.topk_rows_f32(to_dev(x), k, ws=ws)
        rv, ri = oracle.topk_rows_f32(x, k)
        assert_equal_first_diff(to_host(i), ri, f"shared ws call {seed}")
        y = W.scan_i32_full_range(1 << 22, seed=seed)
        assert_equal_first_diff(to_host(ops.scan_inclusive_i32(to_dev(y), ws=ws)),
                                oracle.scan_i32(y), f"scan after topk {seed}")
        kk = W.keys_u32(1 << 22, seed=seed)
        _, p = ops.radix_sort_u32(to_dev(kk.view(np.int32)), ws=ws)
        assert_equal_first_diff(to_host(p), oracle.sort_u32(kk)[1], f"sort after topk {seed}")
    assert ops.workspace_error(ws) == 0


@pytest.mark.parametrize("k", [300, 4096])
@pytest.mark.parametrize("n_top", [16_383, 16_384, 16_385])
@pytest.mark.parametrize("largest", [True, False])
def test_topk_candidate_capacity_edges(ops, n_top, largest, k):
    """Rows of up to 2^17 elements and 256 < k <= 8192 keep the keys whose top
    8 key bits are at least the k-th largest key's, sorted in LDS, when there
    are at most 16384 of them, and are finished the long way otherwise.  Here
    n_top elements of a row share the top key byte of the k-th (values 2 + i
    * 2^-20, all with the same exponent), the rest lie below it (or above it,
    for the smallest k); ties of equal values mixed in.  At k = 4096 the rows
    that fit are finished by two workgroups, one per 2048 ranks."""
    announce("topk capacity edge", n_top, largest, k)
    rows, length = 3, 131_072
    rng = np.random.default_rng(n_top)
    x = np.full((rows, length), 0.5 if largest else 8.0, np.float32)
    for r in range(rows):
        pos = rng.choice(length, n_top, replace=False)
        x[r, pos] = (2.0 + rng.integers(0, 64, n_top) * 2.0**-20).astype(np.float32)
    _check(ops, x, k, largest, f"capacity edge n_top={n_top} largest={largest} k={k}")


@pytest.mark.parametrize("k", [1, 37, 4096, 8192])
def test_topk_long_way_close_values(ops, k):
    """Every key of the row in one top byte (values in [1, 2): one exponent):
    at k = 4096 and 8192 the rows are finished the long way, whose three
    further digit rounds must separate values that differ only in their low
    mantissa bits; at k = 1 and 37 each tile's candidates share the top 16
    bits of its k-th key and the finisher's rounds separate the rest."""
    announce("topk long way", k)
    rng = np.random.default_rng(k)
    x = (1.0 + rng.integers(0, 1 << 23, (4, 65_536)) * 2.0**-23).astype(np.float32)
    x[:, ::97] = x[:, 5:6]  # exact ties across the row
    _check(ops, x, k, True, f"long way k={k}")
    _check(ops, x, k, False, f"long way smallest k={k}")
