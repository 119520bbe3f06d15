"""IEEE special values in the float scans (reading A19: infinities and NaNs
propagate as in IEEE arithmetic).

Whatever the order of the fp32 additions, a running sum is NaN once a NaN or
both infinities precede it, +Inf (-Inf) once only +Inf (-Inf) does, and
finite otherwise; the finite values here are in [-1, 1], far from overflow.
So the NaN positions and the infinities of the GPU result must equal the
oracle's (float64) exactly, and the finite part must be within the float
bound.  Covered: 1-D fp32 inclusive and exclusive (wavefront and register +
LDS tiles), fp16 -> fp32 inclusive on the matrix cores and on the wavefront
tiles, exclusive fp16, the row scans, the reduce-then-scan check variant and
the chunked scans with a carry.
"""
import numpy as np
import pytest

import oracle
from gpu_util import FLOAT_ABS, FLOAT_REL, announce, to_dev, to_host
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu

INF = np.float32(np.inf)
NAN = np.float32(np.nan)


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


def assert_ieee_close(y, ref, absref, what):
    y = np.asarray(y, np.float64).reshape(-1)
    ref, absref = ref.reshape(-1), absref.reshape(-1)
    rn, yn = np.isnan(ref), np.isnan(y)
    if not np.array_equal(rn, yn):
        i = int(np.flatnonzero(rn != yn)[0])
        raise AssertionError(f"{what}: NaN positions differ first at {i}: got {y[i]}, ref {ref[i]}")
    ri = np.isinf(ref)
    if not np.array_equal(y[ri], ref[ri]) or np.isinf(y[~ri & ~rn]).any():
        bad = np.flatnonzero((np.isinf(y) != ri) | (ri & (y != ref)))
        i = int(bad[0])
        raise AssertionError(f"{what}: infinities differ first at {i}: got {y[i]}, ref {ref[i]}")
    f = ~rn & ~ri
    err = np.abs(y[f] - ref[f])
    tol = FLOAT_REL * absref[f] + FLOAT_ABS
    if not (err <= tol).all():
        i = int(np.flatnonzero(f)[np.flatnonzero(~(err <= tol))[0]])
        raise AssertionError(f"{what}: finite value out of tolerance at {i}")


# (name, n, specials as (index, value)): NaN from a NaN on, or from where
# both infinities have been seen; an infinity alone stays.
CASES = [
    ("pos_inf_then_neg_inf", 300_001, [(1000, INF), (150_000, -INF)]),
    ("nan_mid", 300_001, [(70_000, NAN)]),
    ("neg_inf_first_then_pos", 300_001, [(0, -INF), (299_000, INF)]),
    ("two_pos_inf", 300_001, [(5, INF), (123_456, INF)]),
    ("large_tiles", (1 << 27) + 77, [(40_000_000, INF), (90_000_000, NAN)]),
    ("no_special_control", 100_003, []),
]


def _input(n, specials, seed, dtype=np.float32):
    x = W.scan_f32(n, seed=seed).astype(dtype)
    for i, v in specials:
        x[i] = dtype(v)
    return x


@pytest.mark.parametrize("name,n,specials", CASES, ids=[c[0] for c in CASES])
@pytest.mark.parametrize("excl", [False, True])
def test_scan_f32_specials(ops, name, n, specials, excl):
    announce("ieee f32", name, n, excl)
    x = _input(n, specials, seed=n % 1000)
    f = ops.scan_exclusive_f32 if excl else ops.scan_inclusive_f32
    ref, a = oracle.scan_f32(x, exclusive=excl)
    assert_ieee_close(to_host(f(to_dev(x))), ref, a, f"f32 {name} excl={excl}")


@pytest.mark.parametrize("name,n,specials", CASES[:5], ids=[c[0] for c in CASES[:5]])
def test_scan_f16_specials(ops, name, n, specials):
    """fp16 infinities and NaN: the matrix-core kernel must not turn an
    infinity into NaN in the elements before it (inf * 0 in the product)."""
    announce("ieee f16", name, n)
    x = _input(n, specials, seed=n % 997, dtype=np.float16)
    ref, a = oracle.scan_f16(x)
    xd = to_dev(x)
    assert_ieee_close(to_host(ops.scan_inclusive_f16f32(xd)), ref, a, f"f16 {name}")
    assert_ieee_close(to_host(ops.scan_inclusive_f16f32_mfma(xd)), ref, a, f"f16 mfma {name}")
    assert_ieee_close(to_host(ops.scan_inclusive_f16f32_wave(xd)), ref, a, f"f16 wave {name}")
    refe, ae = oracle.scan_f16(x, exclusive=True)
    assert_ieee_close(to_host(ops.scan_exclusive_f16f32(xd)), refe, ae, f"f16 excl {name}")


def test_scan_f16_every_special_pattern(ops):
    """Infinity and NaN bit patterns of fp16 (both infinities, every
    positive-sign NaN payload, three negative ones), each alone in a
    two-tile array; a sample of them through the matrix-core path: NaN from a
    NaN on, the infinity from an infinity."""
    pats = [0x7C00, 0xFC00] + [0x7C00 | p for p in range(1, 1024)] + [0xFC00 | p for p in (1, 512, 1023)]
    n = 32768 * 2
    base = W.scan_f32(n, seed=3).astype(np.float16)
    xs = np.tile(base, (len(pats), 1))
    pos = (np.arange(len(pats)) * 7919) % n
    xs.view(np.uint16)[np.arange(len(pats)), pos] = np.array(pats, np.uint16)
    announce("ieee f16 every special", len(pats))
    xd = to_dev(xs.reshape(-1))
    for r in range(0, len(pats), 97):  # a sample of the rows, each as its own 1-D scan
        y = to_host(ops.scan_inclusive_f16f32_mfma(xd[r * n:(r + 1) * n]))
        ref, a = oracle.scan_f16(xs[r])
        assert_ieee_close(y, ref, a, f"f16 pattern {pats[r]:#06x}")


def test_rows_rss_and_carry_specials(ops):
    announce("ieee rows/rss/carry")
    x = _input(8 * 40_000, [(100, INF), (50_000, NAN), (130_000, -INF), (200_000, INF),
                            (201_000, -INF), (300_000, INF)], seed=5).reshape(8, 40_000)
    ref, a = oracle.scan_rows_f32(x)
    assert_ieee_close(to_host(ops.scan_rows_f32(to_dev(x))), ref, a, "rows")
    flat = x.reshape(-1)
    ref, a = oracle.scan_f32(flat)
    assert_ieee_close(to_host(ops.scan_inclusive_rss_f32(to_dev(flat))), ref, a, "rss")
    # two chunks with the carry between them: an infinity in the first
    # reaches every output of the second through the carry
    h = flat.size // 2
    y1, t1 = ops.scan_inclusive_f32_carry(to_dev(flat[:h]))
    y2, _ = ops.scan_inclusive_f32_carry(to_dev(flat[h:]), carry_in=t1)
    y = np.concatenate([to_host(y1), to_host(y2)])
    assert_ieee_close(y, ref, a, "carry")
