"""GPU parity of the batched row sort, weighted sampling and the top-p sampler
on unsorted rows (through the C ABI), against the oracle.

Row sort: keys bit-exact and in-row indices exact (a stable sort is unique),
special values included.  Samplers: the draw is the oracle's, or lies in the
rounding band around the threshold (the GPU sums in fp32, the oracle in
fp64); rows whose sums are exact in fp32 must match exactly; and, with the
draws theta on a fine grid, the draws reproduce the weights' distribution.
"""
import numpy as np
import pytest

import oracle
from gpu_util import (announce, assert_equal_first_diff, draw_accept, draw_tol, to_dev, to_host,
                      topp_accept)
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


# (3, 200_003): more than 16 tiles per row, so the count table's row scan takes
# the multi-tile (look-back) schedule; (1, 2^20): the 1-D table scan.
SORT_SHAPES = [(1, 1), (3, 5), (1000, 100), (4, 8192), (3, 8193), (7, 10_001),
               (2, 3 * 8192 + 5), (16, 131_072), (3, 200_003), (1, 1 << 20)]


def _row_keys(rows, length, seed):
    k = W.values_f32(rows * length, seed=seed).reshape(rows, length)
    rng = np.random.default_rng(seed)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 1.0, -1.0], np.float32)
    pick = rng.random((rows, length)) < 0.05
    k[pick] = specials[rng.integers(0, specials.size, int(pick.sum()))]
    neg_nan = rng.random((rows, length)) < 0.01
    k[neg_nan] = -np.float32(np.nan)
    return k


@pytest.mark.parametrize("shape", SORT_SHAPES, ids=lambda s: f"{s[0]}x{s[1]}")
@pytest.mark.parametrize("desc", [False, True])
def test_sort_rows_f32(ops, shape, desc):
    rows, length = shape
    announce("sort rows f32", shape, desc)
    k = _row_keys(rows, length, seed=rows + length)
    ko, po = ops.radix_sort_rows_f32(to_dev(k), descending=desc)
    rk, rp = oracle.sort_rows_f32(k, descending=desc)
    assert_equal_first_diff(to_host(ko).view(np.uint32), rk.view(np.uint32), f"keys {shape}")
    assert_equal_first_diff(to_host(po), rp, f"idx {shape}")


def test_sort_rows_keys_only_and_misaligned(ops):
    import torch
    announce("sort rows keys-only / misaligned")
    k = _row_keys(5, 9000, seed=3)
    ko, po = ops.radix_sort_rows_f32(to_dev(k), descending=True, with_perm=False)
    assert po is None
    assert_equal_first_diff(to_host(ko).view(np.uint32),
                            oracle.sort_rows_f32(k, True)[0].view(np.uint32), "keys only")
    flat = to_dev(_row_keys(1, 4 * 8200 + 1, seed=4).reshape(-1))
    view = flat[1:].reshape(4, 8200)  # 4-byte aligned, not 16-byte aligned
    assert view.data_ptr() % 16 != 0
    ko, po = ops.radix_sort_rows_f32(view)
    host = to_host(view)
    rk, rp = oracle.sort_rows_f32(host)
    assert_equal_first_diff(to_host(ko).view(np.uint32), rk.view(np.uint32), "misaligned keys")
    assert_equal_first_diff(to_host(po), rp, "misaligned idx")
    assert ops.radix_sort_rows_f32(torch.empty((0, 5), dtype=torch.float32,
                                               device="cuda"))[0].numel() == 0


# ---------------------------------------------------------------- weighted sampling

def _check_weighted(g, w, theta, what):
    csum, _ = oracle.scan_rows_f32(w)
    ref = oracle.weighted_sample_f32(w, theta)
    bad = []
    for r in range(w.shape[0]):
        if g[r] == ref[r]:
            continue
        total = float(csum[r, -1])
        u = float(theta[r]) * total
        if not draw_accept(int(g[r]), csum[r], u, draw_tol(float(theta[r]), total),
                           w.shape[1] - 1):
            bad.append(r)
    assert not bad, f"{what}: rows {bad[:5]} gpu {g[bad[:5]]} oracle {ref[bad[:5]]}"
    return ref


@pytest.mark.parametrize("length", [1, 3, 64, 4096, 4097, 10_003, 16_384, 16_385, 65_536, 65_537,
                                    131_072, (1 << 20) + 3, 1 << 22, (1 << 22) + 1])
def test_weighted_sample(ops, length):
    """Rows of 4097 to 2^22 take the two-kernel path (4096-element tiles up to
    16384, 8192 above), longer ones the single kernel with per-row arrival."""
    rows = 24 if length < (1 << 20) else 3
    announce("weighted sample", rows, length)
    w = W.sample_weights(rows, length, seed=length)
    theta = W.sample_theta(rows, seed=length)
    g = to_host(ops.weighted_sample_f32(to_dev(w), to_dev(theta)))
    _check_weighted(g, w, theta, f"weighted len={length}")


@pytest.mark.parametrize("length", [5, 4097, 131_072, (1 << 20) + 7])
def test_weighted_sample_exact(ops, length):
    """Integer weights 0..3 and theta in quarters: every fp32 sum and product
    is exact, so the draw must be the oracle's and never a zero weight."""
    rows = 16
    announce("weighted exact", length)
    rng = np.random.default_rng(length)
    w = rng.integers(0, 4, (rows, length)).astype(np.float32)
    w[:, 0] = 1.0
    theta = (rng.integers(0, 4, rows) / 4.0).astype(np.float32)
    g = to_host(ops.weighted_sample_f32(to_dev(w), to_dev(theta)))
    assert_equal_first_diff(g, oracle.weighted_sample_f32(w, theta), f"weighted exact {length}")
    assert all(w[r, g[r]] > 0 for r in range(rows))


def test_weighted_sample_distribution(ops):
    """One weight row repeated with theta on the grid (j + 1/2) / R: token i is
    drawn for a share w_i / W of the grid (inverse transform), so its count is
    R * w_i / W to within one grid step on each side."""
    announce("weighted distribution")
    R, length = 8192, 1000
    w1 = W.sample_weights(1, length, seed=99)
    w = np.repeat(w1, R, axis=0)
    theta = ((np.arange(R) + 0.5) / R).astype(np.float32)
    g = to_host(ops.weighted_sample_f32(to_dev(w), to_dev(theta)))
    counts = np.bincount(g, minlength=length)
    expect = R * w1[0].astype(np.float64) / w1[0].astype(np.float64).sum()
    assert np.all(np.abs(counts - expect) <= 2.0), np.max(np.abs(counts - expect))
    assert counts[w1[0] == 0].sum() == 0


def test_weighted_sample_edges(ops):
    import torch
    announce("weighted edges")
    e = ops.weighted_sample_f32(torch.empty((3, 0), dtype=torch.float32, device="cuda"),
                                to_dev(np.zeros(3, np.float32)))
    assert to_host(e).tolist() == [-1] * 3
    # theta = 0 draws the first non-zero weight; a single non-zero weight is always drawn
    w = np.zeros((4, 70_000), np.float32)
    w[0, 5] = 2.0
    w[1, 69_999] = 1.0
    w[2, 33_333] = 0.5
    w[3, :] = 1.0
    for th in (0.0, 0.5, 0.999):
        theta = np.full(4, th, np.float32)
        g = to_host(ops.weighted_sample_f32(to_dev(w), to_dev(theta)))
        assert g[:3].tolist() == [5, 69_999, 33_333], (th, g)
        assert g[3] == int(np.float64(np.float32(th)) * 70_000), (th, g)


# ---------------------------------------------------------------- top-p sampler

def _check_topp_sample(tok, cut, probs, theta, p, what):
    rows, length = probs.shape
    rt, rc = oracle.topp_sample_f32(probs, theta, p)
    sk, sp = oracle.sort_rows_f32(probs, descending=True)
    bad = []
    for r in range(rows):
        if tok[r] == rt[r] and cut[r] == rc[r]:
            continue
        csum = np.cumsum(sk[r].astype(np.float64))
        k = int(cut[r])
        if not topp_accept(k, int(rc[r]), csum, p):
            bad.append((r, "cutoff"))
            continue
        inv = np.empty(length, np.int64)
        inv[sp[r]] = np.arange(length)
        j = int(inv[tok[r]]) if 0 <= tok[r] < length else -1
        ck = float(csum[k])
        u = float(theta[r]) * ck
        if not draw_accept(j, csum, u, draw_tol(float(theta[r]), ck), k):
            bad.append((r, "token"))
    assert not bad, f"{what}: {bad[:5]} gpu {tok[:5]}/{cut[:5]} oracle {rt[:5]}/{rc[:5]}"
    return rt, rc


@pytest.mark.parametrize("length", [1, 3, 100, 4096, 4097, 10_003, 65_536, 65_537, 131_072,
                                    200_003, 1 << 20, (1 << 20) + 1])
@pytest.mark.parametrize("p", [0.0, 0.5, 0.9, 0.99, 1.5])
def test_topp_sample(ops, length, p):
    """Rows of 4097 to 2^20 draw on the early-exit kernels (the cutoff and the
    draw past the head quarter when p is large), others on the single kernel."""
    rows = 8
    announce("topp sample", rows, length, p)
    probs = W.sample_probs(rows, length, seed=length)
    theta = W.sample_theta(rows, seed=length + 1)
    tok, cut = ops.topp_sample_f32(to_dev(probs), to_dev(theta), p, with_cutoff=True)
    _check_topp_sample(to_host(tok), to_host(cut), probs, theta, p, f"topp sample {length} {p}")


@pytest.mark.parametrize("length", [7, 8192, 70_001, 131_072])
def test_topp_sample_exact(ops, length):
    """Probabilities that are multiples of 2^-24 below 16 * 2^-24, p a dyadic,
    theta in eighths: every fp32 sum and product is exact, ties are many
    (stable order decides), and the GPU must give the oracle's tokens."""
    rows = 16
    announce("topp sample exact", length)
    rng = np.random.default_rng(length)
    probs = (rng.integers(0, 16, (rows, length)) * 2.0**-24).astype(np.float32)
    theta = (rng.integers(0, 8, rows) / 8.0).astype(np.float32)
    total = probs.astype(np.float64).sum(axis=1)
    for frac in (0.25, 0.5, 0.875):
        p = float(np.float32(np.ldexp(np.round(np.ldexp(total.min() * frac, 24)), -24)))
        tok, cut = ops.topp_sample_f32(to_dev(probs), to_dev(theta), p, with_cutoff=True)
        rt, rc = oracle.topp_sample_f32(probs, theta, p)
        assert_equal_first_diff(to_host(cut), rc, f"exact cutoff {length} {frac}")
        assert_equal_first_diff(to_host(tok), rt, f"exact token {length} {frac}")


def test_topp_sample_distribution(ops):
    """One row repeated with theta on a grid: kept token i (in the sorted
    prefix 0..k) is drawn for a share S_i / C_k of the grid; tokens outside
    the nucleus are never drawn."""
    announce("topp distribution")
    R, length, p = 8192, 2000, 0.8
    row = W.sample_probs(1, length, seed=123)
    probs = np.repeat(row, R, axis=0)
    theta = ((np.arange(R) + 0.5) / R).astype(np.float32)
    tok, cut = ops.topp_sample_f32(to_dev(probs), to_dev(theta), p, with_cutoff=True)
    tok, cut = to_host(tok), to_host(cut)
    k = int(oracle.topp_sample_f32(row, theta[:1], p)[1][0])
    assert np.all(cut == cut[0]) and topp_accept(int(cut[0]), k,
                                                 np.cumsum(np.sort(row[0])[::-1]
                                                           .astype(np.float64)), p)
    sk, sp = oracle.sort_rows_f32(row, descending=True)
    kept = sp[0, :int(cut[0]) + 1]
    counts = np.bincount(tok, minlength=length)
    assert counts[np.setdiff1d(np.arange(length), kept)].sum() == 0
    pk = sk[0, :int(cut[0]) + 1].astype(np.float64)
    expect = R * pk / pk.sum()
    assert np.all(np.abs(counts[kept] - expect) <= 2.0), np.max(np.abs(counts[kept] - expect))


def test_topp_sample_edges(ops):
    import torch
    announce("topp sample edges")
    tok, cut = ops.topp_sample_f32(torch.empty((2, 0), dtype=torch.float32, device="cuda"),
                                   to_dev(np.zeros(2, np.float32)), 0.9, with_cutoff=True)
    assert to_host(tok).tolist() == [-1, -1] and to_host(cut).tolist() == [-1, -1]
    # p <= 0 keeps only the most probable token; a one-hot row always gives its token
    probs = W.sample_probs(4, 50_000, seed=8)
    probs[3] = 0.0
    probs[3, 12_345] = 1.0
    theta = np.array([0.0, 0.3, 0.99, 0.7], np.float32)
    tok = to_host(ops.topp_sample_f32(to_dev(probs), to_dev(theta), 0.0))
    assert tok[:3].tolist() == np.argmax(probs[:3], axis=1).tolist()
    assert tok[3] == 12_345


@pytest.mark.parametrize("seed", [0, 1])
def test_topp_sample_config_128x131072(ops, seed):
    announce("topp sample config", seed)
    probs = W.sample_probs(128, 131_072, seed=seed)
    theta = W.sample_theta(128, seed=seed)
    tok, cut = ops.topp_sample_f32(to_dev(probs), to_dev(theta), 0.9, with_cutoff=True)
    _check_topp_sample(to_host(tok), to_host(cut), probs, theta, 0.9, f"config seed={seed}")


def test_weighted_sample_config_128x131072(ops):
    announce("weighted config")
    w = W.sample_probs(128, 131_072, seed=5)
    theta = W.sample_theta(128, seed=5)
    g = to_host(ops.weighted_sample_f32(to_dev(w), to_dev(theta)))
    _check_weighted(g, w, theta, "weighted config")
