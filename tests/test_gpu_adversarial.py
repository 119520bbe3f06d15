"""Adversarial scheduling: every inter-workgroup protocol under random pauses.

libscan_adv.so is the same sources built with LS_ADVERSARIAL_DELAYS: a
pseudo-random pause (usually 0-3 us, one time in eight 14-30 us) after each
tile ticket, before each status-word publication of the decoupled look-back,
and before each row-counter arrival.
Workgroups then reach those steps in orders a normal run seldom produces.
Every op that crosses workgroups runs here against the oracle: the 1-D scans
(wavefront, register + LDS and matrix-core tiles), reduce-then-scan,
compaction, split, the 1-, 4- and 8-bit radix sorts, row scans, both top-p
cutoff kernels, the samplers, the row sort and top-k.
"""
import numpy as np
import pytest

import oracle
from gpu_util import FULL, announce, assert_equal_first_diff, to_dev, to_host, topp_accept
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


@pytest.fixture
def adversarial():
    from paper_2505_15112_amd import _lib
    with _lib.using(_lib.load_adversarial()) as lib:
        yield lib


def test_library_is_the_adversarial_build(ops):
    """Calls are routed to libscan_adv.so inside the block, and its pauses
    are there: the same scan takes clearly longer than with libscan.so."""
    import torch
    from paper_2505_15112_amd import _lib
    announce("adversarial routing")
    x = to_dev(W.scan_i32(1 << 22, seed=3))
    ws = ops.workspace(1, x.device, 1 << 22)
    y = torch.empty_like(x)

    def timed():
        for _ in range(3):
            ops.scan_inclusive_i32(x, out=y, ws=ws)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(20):
            ops.scan_inclusive_i32(x, out=y, ws=ws)
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b)

    plain = timed()
    with _lib.using(_lib.load_adversarial()) as lib:
        assert _lib.load() is lib
        paused = timed()
    assert _lib.load() is not _lib.load_adversarial()
    assert paused > 1.5 * plain, (plain, paused)


@pytest.mark.parametrize("seed", [0, 1])
def test_every_op_on_one_workspace(ops, adversarial, seed):
    """The shared-workspace sequence (scans, reduce-then-scan, compaction,
    split, radix sorts, row scans, both top-p kernels, samplers)."""
    from test_gpu_workspace import _big_ws, _run_all
    announce("adversarial all ops", seed)
    n = 16 * 40_000
    ws = _big_ws(ops, n)
    _run_all(ops, ws, n, 20 + seed)
    assert ops.workspace_error(ws) == 0


@pytest.mark.parametrize("n", [4096 * 3 + 5, (1 << 22) + 7])
def test_scans_mid_sizes(ops, adversarial, n):
    announce("adversarial scans", n)
    x = W.scan_i32_full_range(n, seed=n % 101)
    for excl in (False, True):
        fn = ops.scan_exclusive_i32 if excl else ops.scan_inclusive_i32
        assert_equal_first_diff(to_host(fn(to_dev(x))), oracle.scan_i32(x, exclusive=excl),
                                f"adv i32 n={n} excl={excl}")
    xe = W.exact_pm1(n, seed=5, dtype=np.float16)
    ref = oracle.scan_f16(xe)[0]
    for fn in (ops.scan_inclusive_f16f32, ops.scan_inclusive_f16f32_mfma,
               ops.scan_inclusive_f16f32_wave):
        assert_equal_first_diff(to_host(fn(to_dev(xe))).astype(np.float64), ref,
                                f"adv f16 n={n}")
    b = W.bytes_u8(n, seed=6)
    rb, rt = oracle.scan_u8(b)
    for fn in (ops.scan_exclusive_u8i32, ops.scan_exclusive_u8i32_mfma):
        y, t = fn(to_dev(b))
        assert_equal_first_diff(to_host(y), rb, f"adv u8 n={n}")
        assert int(to_host(t)[0]) == rt


@pytest.mark.skipif(not FULL, reason="full-size cases disabled")
def test_lds_tiles(ops, adversarial):
    """The register + LDS tiles (n >= 2^27), ragged last tile, with carries."""
    import torch
    announce("adversarial lds tiles")
    n = (1 << 27) + 12345
    x = W.scan_i32_full_range(n, seed=61)
    carry = torch.tensor([7], dtype=torch.int32, device="cuda")
    y, _ = ops.scan_exclusive_i32_carry(to_dev(x), carry_in=carry, total_out=carry)
    ref = (oracle.scan_i32(x, exclusive=True).astype(np.int64) + 7).astype(np.int32)
    assert_equal_first_diff(to_host(y), ref, "adv lds")
    assert int(to_host(carry)[0]) == (int(oracle.scan_i32(x)[-1]) + 7 + 2**31) % 2**32 - 2**31


def test_topp_cutoff_and_sampler(ops, adversarial):
    """The cutoff of rows longer than 2^20 (tile sums and a row arrival
    counter; the last tile to arrive decides), on unsorted rows that put the
    crossing anywhere; then the sampler."""
    announce("adversarial topp")
    probs = W.sample_probs(3, (1 << 20) + 4097, seed=8)
    csum, _ = oracle.scan_rows_f32(probs)
    for p in (0.3, 0.9, 1.5):
        g = to_host(ops.topp_cutoff_f32(to_dev(probs), p))
        k = oracle.topp_cutoff_f32(probs, p)
        bad = [r for r in range(3) if not topp_accept(int(g[r]), int(k[r]), csum[r], p)]
        assert not bad, (p, bad)
    rng = np.random.default_rng(9)
    ex = (rng.integers(0, 16, (6, 70_001)) * 2.0**-24).astype(np.float32)
    theta = (rng.integers(0, 8, 6) / 8.0).astype(np.float32)
    tok = to_host(ops.topp_sample_f32(to_dev(ex), to_dev(theta), 2.0**-9))
    assert_equal_first_diff(tok, oracle.topp_sample_f32(ex, theta, 2.0**-9)[0], "adv sampler")


@pytest.mark.parametrize("k,kind", [(64, "normal"), (4096, "normal"), (64, "ties"), (9000, "normal")])
def test_topk(ops, adversarial, k, kind):
    """Top-k's digit rounds (arrival counters), the gather's reservations in
    any order, the long way for rows with too many candidates (ties), and
    the two-chain split (k above 8192)."""
    announce("adversarial topk", k, kind)
    if kind == "ties":
        x = np.random.default_rng(k).integers(-3, 4, (12, 131_072)).astype(np.float32)
    else:
        x = W.values_f32(12 * 131_072, seed=k).reshape(12, 131_072)
    v, i = ops.topk_rows_f32(to_dev(x), k)
    rv, ri = oracle.topk_rows_f32(x, k)
    assert_equal_first_diff(to_host(i), ri, "adv topk indices")
    assert_equal_first_diff(to_host(v).view(np.uint32), rv.view(np.uint32), "adv topk values")
