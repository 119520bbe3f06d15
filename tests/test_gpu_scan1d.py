"""GPU parity of the 1-D scans against the CPU oracle, through the C ABI.

Integers: bit-exact.  Floats: |y - ref| <= 1e-5 * prefix(|x|) + 1e-6 against
the float64 oracle, plus bit-exact runs on {-1, 0, 1} inputs (every partial
sum is an integer far below 2^24, so any summation order is exact).
Sizes span sub-wave, sub-tile, several tiles with ragged tails (tile = 4096
elements), the workloads' full sizes, misaligned views and in-place calls.
"""
import numpy as np
import pytest

import oracle
from gpu_util import (FULL, announce, assert_equal_first_diff, assert_float_close, to_dev,
                      to_host)
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu

SIZES = [1, 2, 63, 64, 65, 255, 256, 257, 1023, 4095, 4096, 4097, 3 * 4096 + 5, 65536,
         (1 << 20) + 17]


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("excl", [False, True])
def test_i32(ops, n, excl):
    announce("i32", n, excl)
    x = W.scan_i32_full_range(n, seed=n)
    fn = ops.scan_exclusive_i32 if excl else ops.scan_inclusive_i32
    y = to_host(fn(to_dev(x)))
    assert_equal_first_diff(y, oracle.scan_i32(x, exclusive=excl), f"i32 n={n}")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("excl", [False, True])
def test_f32(ops, n, excl):
    announce("f32", n, excl)
    x = W.scan_f32(n, seed=n)
    fn = ops.scan_exclusive_f32 if excl else ops.scan_inclusive_f32
    y = to_host(fn(to_dev(x)))
    ref, a = oracle.scan_f32(x, exclusive=excl)
    assert_float_close(y, ref, a, f"f32 n={n}")
    xe = W.exact_pm1(n, seed=n + 1)
    ye = to_host(fn(to_dev(xe)))
    refe, _ = oracle.scan_f32(xe, exclusive=excl)
    assert_equal_first_diff(ye.astype(np.float64), refe, f"f32 exact n={n}")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("excl", [False, True])
def test_f16f32(ops, n, excl):
    announce("f16f32", n, excl)
    x = W.scan_f16(n, seed=n)
    fn = ops.scan_exclusive_f16f32 if excl else ops.scan_inclusive_f16f32
    y = to_host(fn(to_dev(x)))
    ref, a = oracle.scan_f16(x, exclusive=excl)
    assert_float_close(y, ref, a, f"f16 n={n}")
    xe = W.exact_pm1(n, seed=n + 2, dtype=np.float16)
    ye = to_host(fn(to_dev(xe)))
    refe, _ = oracle.scan_f16(xe, exclusive=excl)
    assert_equal_first_diff(ye.astype(np.float64), refe, f"f16 exact n={n}")


@pytest.mark.parametrize("n", SIZES)
def test_u8i32(ops, n):
    announce("u8i32", n)
    x = W.bytes_u8(n, seed=n)
    y, total = ops.scan_exclusive_u8i32(to_dev(x))
    ref, rtot = oracle.scan_u8(x)
    assert_equal_first_diff(to_host(y), ref, f"u8 n={n}")
    assert int(to_host(total)[0]) == rtot


def test_empty(ops):
    import torch
    announce("empty")
    e = torch.empty(0, dtype=torch.int32, device="cuda")
    assert ops.scan_inclusive_i32(e).numel() == 0
    y, tot = ops.scan_exclusive_u8i32(torch.empty(0, dtype=torch.uint8, device="cuda"))
    assert y.numel() == 0 and int(tot.item()) == 0
    cin = torch.tensor([7], dtype=torch.int32, device="cuda")
    _, t = ops.scan_inclusive_i32_carry(e, carry_in=cin)
    assert int(t.item()) == 7


@pytest.mark.parametrize("n", [5, 4097, 100_003])
def test_misaligned_and_inplace(ops, n):
    import torch
    announce("misaligned/inplace", n)
    x = W.scan_i32_full_range(n + 1, seed=3)
    xd = to_dev(x)
    y = torch.empty(n + 1, dtype=torch.int32, device="cuda")
    ops.scan_inclusive_i32(xd[1:], out=y[1:])  # both 4 bytes off 16-byte alignment
    assert_equal_first_diff(to_host(y[1:]), oracle.scan_i32(x[1:]), "misaligned")
    z = xd.clone()
    ops.scan_inclusive_i32(z, out=z)  # in place
    assert_equal_first_diff(to_host(z), oracle.scan_i32(x), "in-place")
    xf = W.scan_f32(n + 1, seed=4)
    yf = ops.scan_exclusive_f32(to_dev(xf)[1:])
    ref, a = oracle.scan_f32(xf[1:], exclusive=True)
    assert_float_close(to_host(yf), ref, a, "misaligned f32")


@pytest.mark.parametrize("excl", [False, True])
def test_carry_chunks(ops, excl):
    """Three chunked calls chained through carry_in / total_out equal one call."""
    import torch
    announce("carry chunks", excl)
    n = 3 * 4096 * 7 + 123
    x = W.scan_i32_full_range(n, seed=9)
    xd = to_dev(x)
    y = torch.empty_like(xd)
    carry = torch.zeros(1, dtype=torch.int32, device="cuda")
    fn = ops.scan_exclusive_i32_carry if excl else ops.scan_inclusive_i32_carry
    cuts = [0, 4096 * 5 + 7, 4096 * 13, n]
    for a, b in zip(cuts[:-1], cuts[1:]):
        fn(xd[a:b], carry_in=carry, out=y[a:b], total_out=carry)
    assert_equal_first_diff(to_host(y), oracle.scan_i32(x, exclusive=excl), "carry chunks")
    assert int(to_host(carry)[0]) == int(oracle.scan_i32(x)[-1])
    xf = W.exact_pm1(n, seed=10)
    xfd = to_dev(xf)
    yf = torch.empty_like(xfd)
    cf = torch.tensor([0.5], dtype=torch.float32, device="cuda")
    fnf = ops.scan_exclusive_f32_carry if excl else ops.scan_inclusive_f32_carry
    for a, b in zip(cuts[:-1], cuts[1:]):
        fnf(xfd[a:b], carry_in=cf, out=yf[a:b], total_out=cf)
    ref, _ = oracle.scan_f32(xf, exclusive=excl)
    assert_equal_first_diff(to_host(yf).astype(np.float64), ref + 0.5, "carry chunks f32")


@pytest.mark.parametrize("n", [1, 4096, 4097, 65536 + 3, (1 << 20) + 17])
def test_rss_matches_lookback(ops, n):
    announce("rss", n)
    x = W.scan_i32_full_range(n, seed=11)
    xd = to_dev(x)
    a = to_host(ops.scan_inclusive_rss_i32(xd))
    b = to_host(ops.scan_inclusive_i32(xd))
    assert_equal_first_diff(a, oracle.scan_i32(x), "rss")
    assert_equal_first_diff(a, b, "rss vs lookback")
    xf = W.scan_f32(n, seed=12)
    yf = to_host(ops.scan_inclusive_rss_f32(to_dev(xf)))
    ref, ab = oracle.scan_f32(xf)
    assert_float_close(yf, ref, ab, "rss f32")


@pytest.mark.parametrize("kind", ["i32", "f32", "f16", "u8"])
@pytest.mark.parametrize("excl", [False, True])
@pytest.mark.parametrize("shift", [0, 1])
def test_large_tiles_ragged(ops, kind, excl, shift):
    """Large-tile schedule (n >= 2^22) with a ragged last tile whose end falls
    inside a lane's 4 elements; shift = 1 runs it on views one element off
    16-byte alignment (the element-wise load/store path)."""
    import torch
    n = (1 << 22) + 3 * 40960 + 12345
    announce("large ragged", kind, excl, shift)
    if kind == "i32":
        x = W.scan_i32_full_range(n + shift, seed=21)
        xd = to_dev(x)[shift:]
        fn = ops.scan_exclusive_i32 if excl else ops.scan_inclusive_i32
        y = torch.empty(n + shift, dtype=torch.int32, device="cuda")
        fn(xd, out=y[shift:])
        assert_equal_first_diff(to_host(y[shift:]), oracle.scan_i32(x[shift:], exclusive=excl), "i32")
    elif kind == "f32":
        x = W.scan_f32(n + shift, seed=22)
        fn = ops.scan_exclusive_f32 if excl else ops.scan_inclusive_f32
        y = torch.empty(n + shift, dtype=torch.float32, device="cuda")
        fn(to_dev(x)[shift:], out=y[shift:])
        ref, a = oracle.scan_f32(x[shift:], exclusive=excl)
        assert_float_close(to_host(y[shift:]), ref, a, "f32")
    elif kind == "f16":
        x = W.exact_pm1(n + shift, seed=23, dtype=np.float16)
        fn = ops.scan_exclusive_f16f32 if excl else ops.scan_inclusive_f16f32
        y = torch.empty(n + shift, dtype=torch.float32, device="cuda")
        fn(to_dev(x)[shift:], out=y[shift:])
        assert_equal_first_diff(to_host(y[shift:]).astype(np.float64),
                                oracle.scan_f16(x[shift:], exclusive=excl)[0], "f16 exact")
    else:
        if not excl:
            pytest.skip("the byte scan is exclusive only")
        x = W.bytes_u8(n + shift, seed=24)
        y, total = ops.scan_exclusive_u8i32(to_dev(x)[shift:])
        ref, rtot = oracle.scan_u8(x[shift:])
        assert_equal_first_diff(to_host(y), ref, "u8")
        assert int(to_host(total)[0]) == rtot


# Register + LDS tiles (n >= 2^27, 16-byte aligned 32-bit data): 114688-element
# integer tiles and 102400-element float tiles; a ragged last tile is scanned
# in passes of 65536.  Sizes: ragged last tiles of one pass (2^27 for integers,
# a last tile of one element) and of two (2^27 for floats, 100000 elements
# past a multiple of the integer tile), and an exact multiple of each tile
# (the last full tile writes the total).
LDS_I32_TILE, LDS_F32_TILE = 114688, 102400
LDS_SIZES = [1 << 27, LDS_I32_TILE * 1170 + 100000, LDS_I32_TILE * 1171,
             LDS_I32_TILE * 1171 + 1, LDS_F32_TILE * 1311, LDS_F32_TILE * 1311 + 1]


@pytest.mark.skipif(not FULL, reason="full-size cases disabled")
@pytest.mark.parametrize("n", LDS_SIZES)
@pytest.mark.parametrize("excl", [False, True])
def test_lds_tiles_i32(ops, n, excl):
    """int32 through the large-array kernel, with carry_in and total_out."""
    import torch
    announce("lds tiles i32", n, excl)
    x = W.scan_i32_full_range(n, seed=31)
    carry = torch.tensor([-123456789], dtype=torch.int32, device="cuda")
    fn = ops.scan_exclusive_i32_carry if excl else ops.scan_inclusive_i32_carry
    y, _ = fn(to_dev(x), carry_in=carry, total_out=carry)
    ref = (oracle.scan_i32(x, exclusive=excl).astype(np.int64) - 123456789).astype(np.int32)
    assert_equal_first_diff(to_host(y), ref, f"lds i32 n={n}")
    tot = (int(oracle.scan_i32(x)[-1]) - 123456789 + 2**31) % 2**32 - 2**31
    assert int(to_host(carry)[0]) == tot


@pytest.mark.skipif(not FULL, reason="full-size cases disabled")
@pytest.mark.parametrize("n", LDS_SIZES)
@pytest.mark.parametrize("excl", [False, True])
def test_lds_tiles_f32(ops, n, excl):
    """fp32 through the large-array kernel: bit-exact on {-1, 0, 1} inputs
    with an exact carry_in, and the total."""
    import torch
    announce("lds tiles f32", n, excl)
    x = W.exact_pm1(n, seed=32)
    cf = torch.tensor([0.5], dtype=torch.float32, device="cuda")
    fn = ops.scan_exclusive_f32_carry if excl else ops.scan_inclusive_f32_carry
    y, _ = fn(to_dev(x), carry_in=cf, total_out=cf)
    ref, _ = oracle.scan_f32(x, exclusive=excl)
    assert_equal_first_diff(to_host(y).astype(np.float64), ref + 0.5, f"lds f32 n={n}")
    assert float(to_host(cf)[0]) == float(np.sum(x.astype(np.float64))) + 0.5


# The matrix-core tile scan (row scans as A * U_32 on MFMA, ScanU): whole
# 32768-element tiles there, the tail on the wavefront kernel.
MFMA_SIZES = [1, 1023, 1024, 32767, 32768, 32769, 3 * 32768 + 12345, (1 << 22) + 5, 1 << 24]


@pytest.mark.parametrize("n", MFMA_SIZES)
def test_wave_f16f32(ops, n):
    """The wavefront-only entry point (the matrix-core path's baseline)."""
    announce("wave f16f32", n)
    x = W.scan_f16(n, seed=n + 5)
    y = to_host(ops.scan_inclusive_f16f32_wave(to_dev(x)))
    ref, a = oracle.scan_f16(x)
    assert_float_close(y, ref, a, f"wave f16 n={n}")


@pytest.mark.parametrize("n", MFMA_SIZES)
def test_mfma_f16f32(ops, n):
    announce("mfma f16f32", n)
    x = W.scan_f16(n, seed=n + 3)
    y = to_host(ops.scan_inclusive_f16f32_mfma(to_dev(x)))
    ref, a = oracle.scan_f16(x)
    assert_float_close(y, ref, a, f"mfma f16 n={n}")
    xe = W.exact_pm1(n, seed=n + 4, dtype=np.float16)
    ye = to_host(ops.scan_inclusive_f16f32_mfma(to_dev(xe)))
    assert_equal_first_diff(ye.astype(np.float64), oracle.scan_f16(xe)[0], f"mfma exact n={n}")


def test_mfma_matches_wavefront_and_repeats(ops):
    """Exact inputs: the matrix-core and wavefront scans agree bit for bit,
    call after call on one workspace (the default path is the matrix-core one)."""
    import torch
    announce("mfma repeat")
    n = 64 * 32768 + 777
    xe = to_dev(W.exact_pm1(n, seed=41, dtype=np.float16))
    ws = ops.workspace(1, xe.device, n)
    ref = ops.scan_inclusive_f16f32_wave(xe, ws=ws)
    assert_equal_first_diff(to_host(ref).astype(np.float64),
                            oracle.scan_f16(to_host(xe))[0], "wave exact")
    assert torch.equal(ops.scan_inclusive_f16f32(xe, ws=ws), ref)
    y = torch.empty_like(ref)
    bad = 0
    for _ in range(20):
        ops.scan_inclusive_f16f32_mfma(xe, out=y, ws=ws)
        bad += int((y != ref).sum().item())
    assert bad == 0


@pytest.mark.parametrize("n", MFMA_SIZES)
def test_mfma_u8i32(ops, n):
    """Bytes 0..255 (the signed MFMA sees x - 128): bit-exact, with the total,
    through the default (wavefront), matrix-core and wavefront entry points."""
    announce("mfma u8", n)
    x = W.bytes_u8(n, seed=n + 6)
    ref, rtot = oracle.scan_u8(x)
    for fn in (ops.scan_exclusive_u8i32, ops.scan_exclusive_u8i32_mfma,
               ops.scan_exclusive_u8i32_wave):
        y, total = fn(to_dev(x))
        assert_equal_first_diff(to_host(y), ref, f"{fn.__name__} n={n}")
        assert int(to_host(total)[0]) == rtot


def test_mfma_u8i32_extremes_and_repeats(ops):
    """All-255 and all-0 bytes (the extremes of the x - 128 correction) and a
    Bernoulli mask, 10 calls each on one workspace."""
    import torch
    announce("mfma u8 extremes")
    n = 40 * 32768 + 99
    ws = ops.workspace(1, torch.device("cuda", 0), n)
    for x in (np.full(n, 255, np.uint8), np.zeros(n, np.uint8), W.mask_u8(n, seed=3)):
        ref, rtot = oracle.scan_u8(x)
        xd = to_dev(x)
        for _ in range(10):
            y, total = ops.scan_exclusive_u8i32_mfma(xd, ws=ws)
            assert_equal_first_diff(to_host(y), ref, "u8 extremes")
            assert int(to_host(total)[0]) == rtot


def test_mfma_rejects_misaligned(ops):
    announce("mfma misaligned")
    x = to_dev(W.scan_f16(1001, seed=5))
    with pytest.raises(Exception):
        ops.scan_inclusive_f16f32_mfma(x[1:])


def test_repeat_no_race(ops):
    """The same input 100 times: the look-back must give one result every time."""
    import torch
    announce("repeat x100")
    n = (1 << 22) + 9
    x = W.scan_i32_full_range(n, seed=13)
    xd = to_dev(x)
    ref = to_dev(oracle.scan_i32(x))
    y = torch.empty_like(xd)
    ws = ops.workspace(1, xd.device, n)
    bad = 0
    for _ in range(100):
        ops.scan_inclusive_i32(xd, out=y, ws=ws)
        bad += int((y != ref).sum().item())
    assert bad == 0


@pytest.mark.skipif(not FULL, reason="full-size cases disabled")
def test_lds_tiles_repeat_no_race(ops):
    """The register + LDS kernel 20 times on one workspace (int32, ragged
    last tile): one result every time."""
    import torch
    announce("lds tiles repeat x20")
    n = (1 << 27) + 12345
    x = W.scan_i32_full_range(n, seed=51)
    xd = to_dev(x)
    ref = to_dev(oracle.scan_i32(x))
    y = torch.empty_like(xd)
    ws = ops.workspace(1, xd.device, n)
    bad = 0
    for _ in range(20):
        ops.scan_inclusive_i32(xd, out=y, ws=ws)
        bad += int((y != ref).sum().item())
    assert bad == 0


@pytest.mark.parametrize("seed", range(6))
def test_random_sizes_and_offsets(ops, seed):
    """Random lengths (up to 2^23) and element offsets through every 1-D
    entry point of the three tile kernels (wavefront, register + LDS at the
    large end is covered above, matrix-core for fp16), against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 1 << 23))
    off = int(rng.integers(0, 8))
    announce("random", seed, n, off)
    xi = W.scan_i32_full_range(n + off, seed=seed)
    assert_equal_first_diff(to_host(ops.scan_inclusive_i32(to_dev(xi)[off:])),
                            oracle.scan_i32(xi[off:]), f"random i32 n={n} off={off}")
    xe = W.exact_pm1(n + off, seed=seed, dtype=np.float16)
    ref = oracle.scan_f16(xe[off:])[0]
    for fn in (ops.scan_inclusive_f16f32, ops.scan_inclusive_f16f32_wave):
        y = to_host(fn(to_dev(xe)[off:]))
        assert_equal_first_diff(y.astype(np.float64), ref, f"random f16 n={n} off={off}")
    if off % 8 == 0:
        y = to_host(ops.scan_inclusive_f16f32_mfma(to_dev(xe)[off:]))
        assert_equal_first_diff(y.astype(np.float64), ref, f"random mfma n={n}")


def test_config_scan_i32_n2_16(ops):
    announce("config i32 n=2^16")
    x = W.scan_i32(1 << 16, seed=0)
    assert_equal_first_diff(to_host(ops.scan_inclusive_i32(to_dev(x))), oracle.scan_i32(x), "c1")


def test_config_f16f32_n2_24(ops):
    announce("config f16f32 n=2^24")
    for seed in (0, 1, 2):
        x = W.scan_f16(1 << 24, seed=seed)
        y = to_host(ops.scan_inclusive_f16f32(to_dev(x)))
        ref, a = oracle.scan_f16(x)
        assert_float_close(y, ref, a, f"c2 seed {seed}")
    xe = W.exact_pm1(1 << 24, seed=5, dtype=np.float16)
    ye = to_host(ops.scan_inclusive_f16f32(to_dev(xe)))
    assert_equal_first_diff(ye.astype(np.float64), oracle.scan_f16(xe)[0], "c2 exact")


@pytest.mark.skipif(not FULL, reason="full-size cases disabled")
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_metric_n2_28_i32(ops, seed):
    announce("metric i32 n=2^28", seed)
    n = W.METRIC_N
    x = W.scan_i32(n, seed=seed)
    y = to_host(ops.scan_inclusive_i32(to_dev(x)))
    assert_equal_first_diff(y, oracle.scan_i32(x), f"metric i32 seed={seed}")


@pytest.mark.skipif(not FULL, reason="full-size cases disabled")
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_metric_n2_28_f32(ops, seed):
    announce("metric f32 n=2^28", seed)
    n = W.METRIC_N
    x = W.scan_f32(n, seed=seed)
    y = to_host(ops.scan_inclusive_f32(to_dev(x)))
    ref, a = oracle.scan_f32(x)
    assert_float_close(y, ref, a, f"metric f32 seed={seed}")
    del ref, a
    if seed:
        return
    xe = W.exact_pm1(n, seed=1)
    ye = to_host(ops.scan_inclusive_f32(to_dev(xe)))
    assert_equal_first_diff(ye.astype(np.float64), oracle.scan_f32(xe)[0], "metric f32 exact")
