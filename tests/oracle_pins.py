"""Pins for the CPU oracle: checks against facts the paper and the mathematics
fix, never against the oracle's own formula.

Each ``check_*`` takes an ``oracle.Oracle`` and raises AssertionError when the
oracle disagrees with
  * the hand-worked fixtures in tests/golden (each cites its passage),
  * closed forms (all-ones, x_i = i, constants, dyadic top-p rows),
  * brute force (O(n^2) sums, exact rational arithmetic) on tiny inputs,
  * Equation (1) of Section 4.1 evaluated with numpy matmuls,
  * independent library routines (numpy cumsum / boolean indexing /
    flatnonzero / stable argsort / searchsorted), and
  * the paper's own algorithms assembled from other oracle functions
    (LSD radix sort from the split oracle).
test_oracle_mutants.py runs the same checks against deliberately broken
builds of oracle.c to show that a dropped term, a wrong sign or index, or a
swapped comparison fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np

from paper_2505_15112_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
M32 = (1 << 32) - 1


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _wrap(v):
    """Python int -> int32 value modulo 2^32."""
    v &= M32
    return v - (1 << 32) if v >= (1 << 31) else v


def _np_cumsum_i32(x):
    return (np.cumsum(x.astype(np.int64)) & M32).astype(np.uint32).view(np.int32)


# ---------------------------------------------------------------- int32 scans

def check_golden_scan_i32(o):
    for c in _golden("scan_int32.json")["cases"]:
        x = np.array(c["x"], np.int32)
        assert o.scan_i32(x).tolist() == c["inclusive"], c
        assert o.scan_i32(x, exclusive=True).tolist() == c["exclusive"], c


def check_scan_i32_bruteforce(o):
    rng = np.random.default_rng(11)
    for n in (1, 2, 3, 17, 64, 65, 200):
        x = W.scan_i32_full_range(n, seed=n)
        xs = [int(v) for v in x]
        inc = [_wrap(sum(xs[: i + 1])) for i in range(n)]
        exc = [_wrap(sum(xs[:i])) for i in range(n)]
        assert o.scan_i32(x).tolist() == inc, n
        assert o.scan_i32(x, exclusive=True).tolist() == exc, n
    del rng


def check_scan_i32_closed_forms(o):
    n = 1 << 17
    i = np.arange(n, dtype=np.int64)
    ones = np.ones(n, np.int32)
    assert np.array_equal(o.scan_i32(ones), (i + 1).astype(np.int32))
    assert np.array_equal(o.scan_i32(ones, exclusive=True), i.astype(np.int32))
    # x_i = i: i(i+1)/2 wraps modulo 2^32 for i >= 92682
    tri = ((i * (i + 1) // 2) & M32).astype(np.uint32).view(np.int32)
    assert np.array_equal(o.scan_i32(i.astype(np.int32)), tri)
    # constant c: c (i+1) mod 2^32
    c = 2**31 - 1
    assert np.array_equal(o.scan_i32(np.full(n, c, np.int32)),
                          ((c * (i + 1)) & M32).astype(np.uint32).view(np.int32))


def check_scan_i32_numpy(o):
    for seed, n in ((0, 1_000_003), (1, 4096)):
        x = W.scan_i32_full_range(n, seed=seed)
        y = o.scan_i32(x)
        assert np.array_equal(y, _np_cumsum_i32(x))
        total = int(x.astype(np.int64).sum()) & M32
        assert int(np.int32(y[-1]).view(np.uint32)) == total
        ye = o.scan_i32(x, exclusive=True)
        assert ye[0] == 0 and np.array_equal(ye[1:], _np_cumsum_i32(x)[:-1])


def check_eq1(o):
    """Equation (1): scan(z) = A U_s + L^-_s A 1_s on zero-padded s x s views."""
    for c in _golden("eq1_tile_scan.json")["cases"]:
        z = np.array(c["z"], np.int32)
        assert o.scan_i32(z).tolist() == c["scan"], c
    rng = np.random.default_rng(5)
    for s in (2, 3, 4, 16, 32):
        for length in (s * s, s * s - 1, (s * s) // 2 + 1):
            z = rng.integers(-1000, 1000, size=length).astype(np.int32)
            A = np.zeros(s * s, np.float64)
            A[:length] = z
            A = A.reshape(s, s)
            U = np.triu(np.ones((s, s)))
            Lm = np.tril(np.ones((s, s)), -1)
            One = np.ones((s, s))
            eq1 = (A @ U + Lm @ A @ One).reshape(-1)[:length]
            assert np.array_equal(o.scan_i32(z).astype(np.float64), eq1), (s, length)


# ---------------------------------------------------------------- float scans

def check_scan_f32_exact_rational(o):
    """Against exact rational prefix sums: the float64 recursive sum of i terms
    is within gamma_i * sum|x| of the exact value (u = 2^-53)."""
    u = 2.0**-53
    for n in (1, 2, 7, 64, 150):
        x = W.scan_f32(n, seed=100 + n)
        for excl in (False, True):
            y, a = o.scan_f32(x, exclusive=excl)
            s = Fraction(0)
            sa = Fraction(0)
            for i in range(n):
                if not excl:
                    s += Fraction(float(x[i]))
                    sa += abs(Fraction(float(x[i])))
                k = i + 1
                gamma = k * u / (1 - k * u)
                assert abs(Fraction(y[i]) - s) <= Fraction(gamma) * sa + Fraction(0), (n, i, excl)
                assert abs(Fraction(a[i]) - sa) <= Fraction(gamma) * sa, (n, i, excl)
                if excl:
                    s += Fraction(float(x[i]))
                    sa += abs(Fraction(float(x[i])))


def check_scan_f32_exact_values(o):
    n = 1_000_001
    x = W.exact_pm1(n, seed=3)
    y, a = o.scan_f32(x)
    xi = x.astype(np.int64)
    assert np.array_equal(y, np.cumsum(xi).astype(np.float64))
    assert np.array_equal(a, np.cumsum(np.abs(xi)).astype(np.float64))
    ye, ae = o.scan_f32(x, exclusive=True)
    assert ye[0] == 0.0 and ae[0] == 0.0
    assert np.array_equal(ye[1:], np.cumsum(xi)[:-1].astype(np.float64))
    # math.fsum gives the correctly rounded total of the whole array
    xr = W.scan_f32(10_000, seed=4)
    yr, _ = o.scan_f32(xr)
    assert abs(yr[-1] - math.fsum(float(v) for v in xr)) <= 1e4 * 2.0**-53 * 1e4


def check_f16_decode_all(o):
    for c in _golden("fp16_values.json")["cases"]:
        v = o.half_to_double(int(c["bits"], 16))
        want = float(c["value"])
        if math.isnan(want):
            assert math.isnan(v), c
        else:
            assert v == want and math.copysign(1, v) == math.copysign(1, want), c
    bits = np.arange(1 << 16, dtype=np.uint16)
    ref = bits.view(np.float16).astype(np.float64)
    got = np.array([o.half_to_double(int(b)) for b in bits])
    nan = np.isnan(ref)
    assert np.array_equal(nan, np.isnan(got))
    assert np.array_equal(ref[~nan], got[~nan])
    assert np.array_equal(np.signbit(ref[~nan]), np.signbit(got[~nan]))


def check_scan_f16(o):
    x = W.exact_pm1(100_003, seed=8, dtype=np.float16)
    y, a = o.scan_f16(x)
    xi = x.astype(np.int64)
    assert np.array_equal(y, np.cumsum(xi).astype(np.float64))
    assert np.array_equal(a, np.cumsum(np.abs(xi)).astype(np.float64))
    # dyadic fp16 values: every partial sum is exact in float64
    xh = W.scan_f16(4096, seed=9)
    y, _ = o.scan_f16(xh)
    exact = np.cumsum([Fraction(float(v)) for v in xh.astype(np.float64)])
    assert all(Fraction(float(yv)) == e for yv, e in zip(y, exact))
    ye, _ = o.scan_f16(xh, exclusive=True)
    assert ye[0] == 0.0 and all(Fraction(float(yv)) == e for yv, e in zip(ye[1:], exact[:-1]))


def check_scan_u8(o):
    for c in _golden("scan_u8.json")["cases"]:
        y, t = o.scan_u8(np.array(c["x"], np.uint8))
        assert y.tolist() == c["exclusive"] and t == c["total"], c
    x = W.bytes_u8(1_000_000, seed=2)
    y, t = o.scan_u8(x)
    cs = np.cumsum(x.astype(np.int64))
    assert y[0] == 0 and np.array_equal(y[1:].astype(np.int64), cs[:-1])
    assert t == int(cs[-1])
    yi = o.scan_u8(x, exclusive=False)
    assert np.array_equal(yi.astype(np.int64), cs)


# ---------------------------------------------------------------- batched rows

def check_rows(o):
    rows, length = 7, 1000
    ones = np.ones((rows, length), np.int32)
    want = np.tile(np.arange(1, length + 1, dtype=np.int32), (rows, 1))
    assert np.array_equal(o.scan_rows_i32(ones), want)
    assert np.array_equal(o.scan_rows_i32(ones, exclusive=True), want - 1)
    x = W.scan_i32_full_range(rows * length, seed=6).reshape(rows, length)
    y = o.scan_rows_i32(x)
    for r in range(rows):
        assert np.array_equal(y[r], _np_cumsum_i32(x[r]))
    xf = W.exact_pm1(rows * length, seed=7).reshape(rows, length)
    yf, af = o.scan_rows_f32(xf)
    assert np.array_equal(yf, np.cumsum(xf.astype(np.int64), axis=1).astype(np.float64))
    assert np.array_equal(af, np.cumsum(np.abs(xf.astype(np.int64)), axis=1).astype(np.float64))
    ye, _ = o.scan_rows_f32(xf, exclusive=True)
    assert np.all(ye[:, 0] == 0) and np.array_equal(ye[:, 1:], yf[:, :-1])


# ---------------------------------------------------------------- compaction / split

def check_compact(o):
    for c in _golden("compress_split.json")["compress"]:
        out, idx = o.compact_f32(np.array(c["x"], np.float32), np.array(c["mask"], np.uint8))
        assert out.tolist() == c["out"] and idx.tolist() == c["idx"], c
    n = 300_001
    x = W.values_f32(n, seed=1)
    m = W.mask_u8(n, seed=1)
    m[::7] = 200  # non-0/1 bytes count as true
    out, idx = o.compact_f32(x, m)
    keep = m.astype(bool)
    assert np.array_equal(idx, np.flatnonzero(keep).astype(np.int32))
    assert np.array_equal(out.view(np.uint32), x[keep].view(np.uint32))


def check_split(o):
    for c in _golden("compress_split.json")["split"]:
        ko, io, nt = o.split_u32(np.array(c["keys"], np.uint32), np.array(c["flags"], np.uint8))
        assert ko.tolist() == c["keys_out"] and io.tolist() == c["idx_out"], c
        assert nt == c["n_true"], c
    n = 200_003
    k = W.keys_u32(n, seed=2)
    f = W.mask_u8(n, seed=2)
    ko, io, nt = o.split_u32(k, f)
    order = np.concatenate([np.flatnonzero(f), np.flatnonzero(f == 0)]).astype(np.int32)
    assert nt == int(f.sum())
    assert np.array_equal(io, order) and np.array_equal(ko, k[order])
    perm = np.random.default_rng(3).permutation(n).astype(np.int32)
    ko, io, nt = o.split_u32(k, f, idx_in=perm)
    assert np.array_equal(io, perm[order]) and np.array_equal(ko, k[order])


# ---------------------------------------------------------------- sort

def _check_sorted(keys, ko, perm):
    n = keys.size
    assert np.array_equal(np.sort(perm), np.arange(n, dtype=np.int32))
    assert np.array_equal(ko, keys[perm])
    assert np.all(ko[1:] >= ko[:-1])
    same = ko[1:] == ko[:-1]
    assert np.all(perm[1:][same] > perm[:-1][same])  # stable


def check_sort(o):
    for c in _golden("radix_sort.json")["cases"]:
        ko, perm = o.sort_u32(np.array(c["keys"], np.uint32))
        assert ko.tolist() == c["sorted"] and perm.tolist() == c["perm"], c
    for keys in (W.keys_u32(300_000, seed=4), W.keys_u32(100_000, seed=5) % np.uint32(16),
                 np.zeros(1000, np.uint32)):
        ko, perm = o.sort_u32(keys)
        _check_sorted(keys, ko, perm)
        ref = np.argsort(keys, kind="stable").astype(np.int32)
        assert np.array_equal(perm, ref)


def check_sort_lsd_split(o):
    """Section 5 'Radix Sort': 32 stable splits, least significant bit first,
    with flag = NOT bit (zeros go first), reach the oracle's sorted order; so
    does a stable LSD pass per 4-bit digit (numpy stable argsort per digit)."""
    keys = W.keys_u32(20_000, seed=6)
    keys[::3] %= np.uint32(64)  # plenty of equal keys
    k = keys.copy()
    idx = np.arange(keys.size, dtype=np.int32)
    for b in range(32):
        flags = (((k >> np.uint32(b)) & np.uint32(1)) == 0).astype(np.uint8)
        k, idx, _ = o.split_u32(k, flags, idx_in=idx)
    ko, perm = o.sort_u32(keys)
    assert np.array_equal(k, ko) and np.array_equal(idx, perm)
    k4 = keys.copy()
    idx4 = np.arange(keys.size, dtype=np.int32)
    for d in range(8):
        digit = (k4 >> np.uint32(4 * d)) & np.uint32(15)
        order = np.argsort(digit, kind="stable")
        k4, idx4 = k4[order], idx4[order]
    assert np.array_equal(k4, ko) and np.array_equal(idx4, perm)


def check_sort_typed_golden(o):
    g = _golden("sort_typed.json")
    for c in g["i32"]:
        k = np.array(c["keys"], np.int32)
        for desc, key in ((False, "asc_perm"), (True, "desc_perm")):
            ko, perm = o.sort_i32(k, descending=desc)
            assert perm.tolist() == c[key] and np.array_equal(ko, k[perm]), (desc, perm)
    for name, dt, bt in (("f32_bits", np.float32, np.uint32), ("f16_bits", np.float16, np.uint16)):
        for c in g[name]:
            bits = np.array([int(h, 16) for h in c["keys"]], bt)
            fn = o.sort_f32 if dt is np.float32 else o.sort_f16
            for desc, key in ((False, "asc_perm"), (True, "desc_perm")):
                ko, perm = fn(bits.view(dt), descending=desc)
                assert perm.tolist() == c[key], (name, desc, perm)
                assert np.array_equal(ko.view(bt), bits[perm]), (name, desc)


def check_sort_typed_numpy(o):
    """Against numpy's stable argsort (ascending, and on the negated keys for
    descending) where numpy's order is the same: integers, and floats with no
    NaN and no -0 (numpy ranks -0 and +0 equal)."""
    rng = np.random.default_rng(17)
    ki = rng.integers(-2**31, 2**31, 50_000, dtype=np.int64).astype(np.int32)
    ki[::7] = ki[::7] % 5  # ties
    ki[:4] = [-2**31, 2**31 - 1, 0, -1]
    for desc in (False, True):
        ko, perm = o.sort_i32(ki, descending=desc)
        ref = np.argsort(-ki.astype(np.int64) if desc else ki, kind="stable").astype(np.int32)
        assert np.array_equal(perm, ref) and np.array_equal(ko, ki[perm]), desc
    for dt in (np.float32, np.float16):
        kf = (rng.standard_normal(40_000) * 100).astype(dt)
        kf[::5] = np.round(kf[::5] / 10) * 10  # ties
        kf[kf == 0] = dt(1)  # no zeros of either sign
        kf[:3] = [np.inf, -np.inf, dt(-2.5)]
        fn = o.sort_f32 if dt is np.float32 else o.sort_f16
        for desc in (False, True):
            ko, perm = fn(kf, descending=desc)
            ref = np.argsort(-kf if desc else kf, kind="stable").astype(np.int32)
            assert np.array_equal(perm, ref), (dt, desc)
            assert np.array_equal(ko, kf[perm]), (dt, desc)


def check_sort_rows(o):
    """Each row equals numpy's stable argsort of that row (finite, no -0)."""
    rng = np.random.default_rng(23)
    x = (rng.standard_normal((7, 1000)) * 10).astype(np.float32)
    x[:, ::4] = np.round(x[:, ::4])
    x[x == 0] = 1.0
    for desc in (False, True):
        ko, idx = o.sort_rows_f32(x, descending=desc)
        for r in range(x.shape[0]):
            ref = np.argsort(-x[r] if desc else x[r], kind="stable")
            assert np.array_equal(idx[r], ref) and np.array_equal(ko[r], x[r][ref]), (r, desc)


def check_weighted_sample(o):
    """Appendix "Weighted Sampling": equal weights give floor(theta * len) in
    closed form; random weights match numpy's searchsorted(side='right') on
    the float64 cumulative sum."""
    for length in (1, 7, 1000):
        th = np.array([0.0, 0.25, 0.5, 0.999, 0.3], np.float32)
        w = np.ones((th.size, length), np.float32)
        got = o.weighted_sample_f32(w, th)
        want = np.minimum(np.floor(th.astype(np.float64) * length), length - 1).astype(np.int32)
        assert np.array_equal(got, want), (length, got, want)
    rng = np.random.default_rng(29)
    w = rng.random((50, 300)).astype(np.float32)
    w[:, ::3] = 0  # zero weights are never drawn
    th = rng.random(50).astype(np.float32)
    got = o.weighted_sample_f32(w, th)
    for r in range(50):
        c = np.cumsum(w[r].astype(np.float64))
        j = int(np.searchsorted(c, float(th[r]) * c[-1], side="right"))
        assert got[r] == min(j, 299) and w[r, got[r]] > 0, r


def check_topp_sample(o):
    """The top-p sampler against a numpy composition of its definition:
    stable descending argsort, float64 cumulative sum, searchsorted cutoff,
    inverse-transform draw among the kept tokens."""
    rng = np.random.default_rng(31)
    probs = W.topp_probs(40, 2048, seed=3)
    probs = np.stack([r[rng.permutation(r.size)] for r in probs])  # unsorted rows
    th = rng.random(40).astype(np.float32)
    for p in (0.9, 0.5, 1e-9, 1.5):
        tok, cut = o.topp_sample_f32(probs, th, p)
        pf = float(np.float32(p))
        for r in range(40):
            order = np.argsort(-probs[r], kind="stable")
            c = np.cumsum(probs[r][order].astype(np.float64))
            k = min(int(np.searchsorted(c, pf, side="left")), 2047)
            j = min(int(np.searchsorted(c[: k + 1], float(th[r]) * c[k], side="right")), k)
            assert cut[r] == k and tok[r] == order[j], (p, r)
    # a hand-worked row: probabilities 0.1 0.4 0.2 0.3, p = 0.65 keeps the
    # sorted tokens 1 (0.4) and 3 (0.3) (0.4 + 0.3 = 0.7 >= 0.65); theta = 0.6
    # draws from C = 0.4, 0.7 at u = 0.42: the second kept token, 3.
    tok, cut = o.topp_sample_f32(np.array([[0.1, 0.4, 0.2, 0.3]], np.float32),
                                 np.array([0.6], np.float32), 0.65)
    assert cut.tolist() == [1] and tok.tolist() == [3], (tok, cut)


# ---------------------------------------------------------------- top-k

def _bits(hexes):
    return np.array([int(h, 16) for h in hexes], np.uint32)


def check_topk_golden(o):
    """Section 5 "Top-k": hand-worked rows with ties, signed zeros, infinities
    and NaNs of both signs, both directions, k = 0 and k = len."""
    for c in _golden("topk.json")["cases"]:
        x = _bits(c["x"]).view(np.float32).reshape(1, -1)
        v, i = o.topk_rows_f32(x, c["k"], largest=c["largest"])
        assert v.view(np.uint32).reshape(-1).tolist() == _bits(c["values"]).tolist(), c["why"]
        assert i.reshape(-1).tolist() == c["idx"], c["why"]


def _totalorder_key(bits):
    """Unsigned key whose order is IEEE 754 totalOrder on binary32 patterns."""
    b = bits.astype(np.uint64)
    return np.where(b >> 31, (~b) & 0xFFFFFFFF, b | 0x80000000)


def check_topk_bruteforce(o):
    """The definition by counting, on tiny rows with many ties: element i is
    kept iff fewer than k elements come before it in the stable order (larger
    values, or equal values at lower indices); the kept ones are listed by
    that rank."""
    rng = np.random.default_rng(37)
    for trial in range(40):
        length = int(rng.integers(1, 12))
        x = rng.integers(-3, 4, (2, length)).astype(np.float32)
        x[x == 0] = rng.choice(np.array([0.0, -0.0], np.float32), int((x == 0).sum()))
        k = int(rng.integers(0, length + 1))
        for largest in (True, False):
            v, idx = o.topk_rows_f32(x, k, largest=largest)
            for r in range(2):
                key = _totalorder_key(x[r].view(np.uint32))
                if not largest:
                    key = (~key) & 0xFFFFFFFF
                rank = [sum(1 for j in range(length)
                            if key[j] > key[i] or (key[j] == key[i] and j < i))
                        for i in range(length)]
                want = sorted((i for i in range(length) if rank[i] < k), key=lambda i: rank[i])
                assert idx[r].tolist() == want, (trial, largest, r)
                assert v[r].view(np.uint32).tolist() == x[r].view(np.uint32)[want].tolist()


def check_topk_numpy(o):
    """numpy's stable argsort of the totalOrder key (complemented for the
    largest) gives the same indices; values are the row's bits at them."""
    rng = np.random.default_rng(41)
    x = rng.standard_normal((6, 3000)).astype(np.float32)
    x[:, ::7] = np.round(x[:, ::7])  # ties
    x[1, 5] = np.float32(np.nan)
    x[2, 9] = -np.float32(np.inf)
    for k in (1, 17, 3000):
        for largest in (True, False):
            v, idx = o.topk_rows_f32(x, k, largest=largest)
            for r in range(6):
                key = _totalorder_key(x[r].view(np.uint32)).astype(np.int64)
                order = np.argsort(-key if largest else key, kind="stable")[:k]
                assert np.array_equal(idx[r], order), (k, largest, r)
                assert np.array_equal(v[r].view(np.uint32), x[r].view(np.uint32)[order])


# ---------------------------------------------------------------- top-p

def check_topp(o):
    for c in _golden("topp.json")["cases"]:
        cut = o.topp_cutoff_f32(np.array([c["probs"]], np.float32), c["p"])
        assert cut.tolist() == [c["cutoff"]], c
    # closed form: 2^m equal probabilities 2^-m, p = 1/2 -> index 2^(m-1) - 1
    for m in (1, 4, 10, 17):
        probs = np.full((2, 1 << m), 2.0**-m, np.float32)
        assert o.topp_cutoff_f32(probs, 0.5).tolist() == [(1 << (m - 1)) - 1] * 2
    probs = W.topp_probs(16, 4096, seed=1)
    for p in (0.9, 0.5, 0.999, 1e-9):
        cut = o.topp_cutoff_f32(probs, p)
        pf = float(np.float32(p))
        for r in range(probs.shape[0]):
            cs = np.cumsum(probs[r].astype(np.float64))
            k = int(np.searchsorted(cs, pf, side="left"))
            assert cut[r] == min(k, probs.shape[1] - 1), (p, r)




# ---------------------------------------------------------------- IEEE special values

def _same_ieee(got, want):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    return got.shape == want.shape and bool(np.all((got == want) | (np.isnan(got) & np.isnan(want))))


def check_scan_float_ieee_specials(o):
    """Reading A19: infinities and NaNs propagate as in IEEE arithmetic.  The
    expected running sums are Python's own (IEEE double) sequential sums."""
    inf, nan = float("inf"), float("nan")
    for xs in ([0.5, inf, 0.25, -inf, 1.0], [-inf, 1.0, -inf, 2.0], [1.0, nan, 2.0, inf],
               [inf, inf, -1.0], [0.0, -0.0, -inf, inf]):
        inc, exc, acc = [], [], 0.0
        for v in xs:
            exc.append(acc)
            acc += v
            inc.append(acc)
        for dt, scan in ((np.float32, o.scan_f32), (np.float16, o.scan_f16)):
            x = np.array(xs, dt)
            y, _ = scan(x)
            assert _same_ieee(y, inc), (dt, xs, y, inc)
            y, _ = scan(x, exclusive=True)
            assert _same_ieee(y, exc), (dt, xs, y, exc)
        y, _ = o.scan_rows_f32(np.array([xs, xs[::-1]], np.float32))
        back = []
        acc = 0.0
        for v in xs[::-1]:
            acc += v
            back.append(acc)
        assert _same_ieee(y[0], inc) and _same_ieee(y[1], back), (xs, y)


ALL_CHECKS = [v for k, v in sorted(globals().items()) if k.startswith("check_")]
