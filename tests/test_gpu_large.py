"""The C ABI's documented size limits, exercised at or past them on the GPU.

- 1-D scans: int32 at n = 2^35 (the limit, in place: 128 GiB) and at
  2^31 + 12345, fp32 at 2^31 + 5, the exclusive byte scan at 2^31 + 777
  (64-bit element offsets past 2^31, tile counts far past any other test).
- Compaction and split at n = INT32_MAX (their limit: int32 positions, counts
  and indices).
- The 8-, 4- and 1-bit radix sorts at n = INT32_MAX keys with the permutation
  (count-table offsets past 2^30 and 2^31 - 1 output positions).
- Weighted sampling and the top-p sampler on one row of 2^25 + 3 elements
  (the paper's arbitrary support size, past the 2^24 its baseline allows).

At these sizes the inputs are generated on the GPU from a closed form (a
multiplicative hash of the index), and the results are checked chunk by chunk
on the GPU against properties that determine them uniquely: the scan's
recursion y_i = y_(i-1) + x_i (exclusive: + x_(i-1)) with its first value;
for compaction, that the indices are strictly increasing, all flagged and as
many as there are flags, and that each value is its source's bits; for the
split, that the indices are a permutation with the flagged ones first, each
part in index order; for a sort, that the keys are non-decreasing, the
permutation is a permutation, keys_out = keys[perm] and equal keys keep index
order.  The samplers are checked against the oracle (host), within the
acceptance band of the float readings.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, draw_accept, draw_tol, to_dev, to_host, topp_accept
from paper_2505_15112_amd import workloads as W

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

CHUNK = 1 << 28
INT32_MAX = (1 << 31) - 1


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


@pytest.fixture(autouse=True)
def _release():
    import torch
    torch.cuda.empty_cache()
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _need(nbytes):
    import torch
    free, _ = torch.cuda.mem_get_info()
    if free < nbytes:
        pytest.skip(f"needs {nbytes / 2**30:.0f} GiB of free device memory, {free / 2**30:.0f} free")


def _hash(start, stop, salt=0):
    """h(i) = (i * 2654435761 + salt) mod 2^32 for i in [start, stop), int64."""
    import torch
    i = torch.arange(start, stop, dtype=torch.int64, device="cuda")
    return (((i & 0xFFFFFFFF) * 2654435761 + salt) & 0xFFFFFFFF)


def _fill(t, fn):
    """t[s:e] = fn(s, e) chunk by chunk (fn returns a tensor of t's dtype)."""
    n = t.numel()
    for s in range(0, n, CHUNK):
        e = min(n, s + CHUNK)
        t[s:e] = fn(s, e)


def _check_recursion(y, x_of, exclusive, first, what):
    """y_0 == first and y_i - y_(i-1) == x_(i-1 if exclusive else i), chunked."""
    import torch
    n = y.numel()
    assert y[0].item() == first, (what, y[0].item(), first)
    for s in range(1, n, CHUNK):
        e = min(n, s + CHUNK)
        d = y[s:e] - y[s - 1:e - 1]
        want = x_of(s - 1, e - 1) if exclusive else x_of(s, e)
        bad = torch.nonzero(d != want)
        if bad.numel():
            i = s + int(bad[0, 0])
            raise AssertionError(f"{what}: recursion broken at {i}: got {y[i].item()} after "
                                 f"{y[i - 1].item()}")


def test_scan_i32_at_2p35_in_place(ops):
    """The largest 1-D scan the ABI accepts, in place: x_i = i mod 2^32, so
    the recursion pins every output (and y_i = i(i+1)/2 mod 2^32)."""
    import torch
    n = 1 << 35
    _need(n * 4 + (24 << 30))
    announce("scan_inclusive_i32 in place", n)
    x = torch.empty(n, dtype=torch.int32, device="cuda")
    iota = lambda s, e: torch.arange(s, e, dtype=torch.int64, device="cuda").to(torch.int32)  # noqa: E731
    _fill(x, iota)
    ops.scan_inclusive_i32(x, out=x)
    torch.cuda.synchronize()
    _check_recursion(x, iota, False, 0, "i32 2^35")
    for i in (1 << 31, (1 << 33) + 3, n - 1):  # closed form at a few indices (Python integers)
        assert int(x[i].item()) % 2**32 == (i * (i + 1) // 2) % 2**32, i


def test_scan_i32_past_2p31(ops):
    """x_i in 0..100 (hashed), n = 2^31 + 12345, out of place."""
    import torch
    n = (1 << 31) + 12345
    _need(n * 8 + (8 << 30))
    announce("scan_inclusive_i32", n)
    xv = lambda s, e: ((_hash(s, e) >> 8) % 101).to(torch.int32)  # noqa: E731
    x = torch.empty(n, dtype=torch.int32, device="cuda")
    _fill(x, xv)
    y = ops.scan_inclusive_i32(x)
    torch.cuda.synchronize()
    _check_recursion(y, xv, False, int(x[0].item()), "i32 2^31+12345")


def test_scan_f32_exact_past_2p31(ops):
    """x_i in {-1, 0, 1} (hashed), n = 2^31 + 5: every running sum is an
    integer of magnitude below 2^23 (checked), so the sum of any contiguous
    range stays below 2^24, every fp32 sum is exact in any order and the
    recursion must hold exactly."""
    import torch
    n = (1 << 31) + 5
    _need(n * 8 + (8 << 30))
    announce("scan_inclusive_f32 exact", n)
    xv = lambda s, e: ((_hash(s, e, 12345) >> 11) % 3 - 1).to(torch.float32)  # noqa: E731
    x = torch.empty(n, dtype=torch.float32, device="cuda")
    _fill(x, xv)
    # the input's running sums stay below 2^23 in magnitude (exactness holds)
    carry, peak = 0, 0
    for s in range(0, n, CHUNK):
        c = torch.cumsum(x[s:min(n, s + CHUNK)].to(torch.int64), 0) + carry
        peak = max(peak, int(c.abs().max().item()))
        carry = int(c[-1].item())
    assert peak < 2**23, peak
    y = ops.scan_inclusive_f32(x)
    torch.cuda.synchronize()
    _check_recursion(y, xv, False, float(x[0].item()), "f32 2^31+5")


def test_scan_u8_exclusive_past_2p31(ops):
    """Bytes 0..255 (hashed), n = 2^31 + 777, with the total."""
    import torch
    n = (1 << 31) + 777
    _need(n * 5 + (8 << 30))
    announce("scan_exclusive_u8i32", n)
    xv = lambda s, e: (_hash(s, e, 99) >> 24).to(torch.uint8)  # noqa: E731
    x = torch.empty(n, dtype=torch.uint8, device="cuda")
    _fill(x, xv)
    y, total = ops.scan_exclusive_u8i32(x)
    torch.cuda.synchronize()
    _check_recursion(y, lambda s, e: xv(s, e).to(torch.int32), True, 0, "u8 2^31+777")
    want = (int(y[-1].item()) + int(x[-1].item()) + 2**31) % 2**32 - 2**31
    assert int(total.item()) == want


def _mask(s, e):
    import torch
    return ((_hash(s, e, 7) >> 13) & 1).to(torch.uint8)


def test_compact_at_int32_max(ops):
    """n = INT32_MAX values whose bits are their index, half of them kept."""
    import torch
    n = INT32_MAX
    _need(n * 13 + (8 << 30))
    announce("compact_by_mask_f32", n)
    xi = torch.empty(n, dtype=torch.int32, device="cuda")
    _fill(xi, lambda s, e: torch.arange(s, e, dtype=torch.int32, device="cuda"))
    m = torch.empty(n, dtype=torch.uint8, device="cuda")
    _fill(m, _mask)
    out, idx, cnt = ops.compact_by_mask_f32(xi.view(torch.float32), m, with_idx=True)
    torch.cuda.synchronize()
    c = int(cnt.item())
    flagged = sum(int(m[s:s + CHUNK].sum(dtype=torch.int64).item()) for s in range(0, n, CHUNK))
    assert c == flagged, (c, flagged)
    oi = out.view(torch.int32)
    for s in range(0, c, CHUNK):
        e = min(c, s + CHUNK)
        ic = idx[s:e]
        assert bool(torch.equal(oi[s:e], ic)), ("values are not their sources' bits", s)
        assert bool((m[ic.long()] != 0).all()), ("an unflagged index was kept", s)
        lo = idx[max(0, s - 1):e]
        assert bool((lo[1:] > lo[:-1]).all()), ("indices not strictly increasing", s)


def test_split_at_int32_max(ops):
    """n = INT32_MAX keys equal to their index: flagged first, each part in
    index order, indices a permutation."""
    import torch
    n = INT32_MAX
    _need(n * 15 + (8 << 30))
    announce("split_by_flags_u32", n)
    keys = torch.empty(n, dtype=torch.int32, device="cuda")
    _fill(keys, lambda s, e: torch.arange(s, e, dtype=torch.int32, device="cuda"))
    f = torch.empty(n, dtype=torch.uint8, device="cuda")
    _fill(f, _mask)
    ko, io, nt = ops.split_by_flags_u32(keys, f)
    torch.cuda.synchronize()
    t = int(nt.item())
    flagged = sum(int(f[s:s + CHUNK].sum(dtype=torch.int64).item()) for s in range(0, n, CHUNK))
    assert t == flagged, (t, flagged)
    assert bool(torch.equal(ko, io)), "keys did not move with their indices"
    seen = torch.zeros(n, dtype=torch.uint8, device="cuda")
    for s in range(0, n, CHUNK):
        e = min(n, s + CHUNK)
        ic = io[s:e].long()
        seen.index_fill_(0, ic, 1)
        fl = f[ic] != 0
        if e <= t:
            assert bool(fl.all()), ("unflagged key in the flagged part", s)
        elif s >= t:
            assert bool((~fl).all()), ("flagged key in the other part", s)
        else:
            assert bool(fl[:t - s].all()) and bool((~fl[t - s:]).all()), ("parts", s)
        lo = io[max(0, s - 1):e]
        inc = lo[1:] > lo[:-1]
        if s - 1 < t <= e - 1 and t > 0:  # the boundary between the parts
            inc[t - max(0, s - 1) - 1] = True
        assert bool(inc.all()), ("a part is not in index order", s)
    assert bool((seen != 0).all()), "indices are not a permutation"


def _check_sorted(keys, ko, po, what):
    """Stable ascending uint32 sort of keys (int32 views): unique result."""
    import torch
    n = keys.numel()
    sign = torch.tensor(-2**31, dtype=torch.int32, device="cuda")
    seen = torch.zeros(n, dtype=torch.uint8, device="cuda")
    for s in range(0, n, CHUNK):
        e = min(n, s + CHUNK)
        pc = po[s:e].long()
        seen.index_fill_(0, pc, 1)
        assert bool(torch.equal(keys[pc], ko[s:e])), (what, "keys_out != keys[perm]", s)
        lo = max(0, s - 1)
        a, b = ko[lo:e - 1] ^ sign, ko[lo + 1:e] ^ sign  # unsigned order as signed
        assert bool((b >= a).all()), (what, "not sorted", s)
        eq = b == a
        pa, pb = po[lo:e - 1], po[lo + 1:e]
        assert bool((pb[eq] > pa[eq]).all()), (what, "equal keys out of index order", s)
    assert bool((seen != 0).all()), (what, "perm is not a permutation")


def test_radix_sorts_at_int32_max(ops):
    """INT32_MAX hashed 32-bit keys with 2^12 copies of each 20-bit value in
    the low half of the range (stability exercised): 8-bit digits checked by
    the sort properties, 4- and 1-bit digits equal to it bit for bit."""
    import torch
    n = INT32_MAX
    _need(n * 28 + (10 << 30))
    announce("radix_sort_u32 8-bit", n)
    keys = torch.empty(n, dtype=torch.int32, device="cuda")
    # half the keys full 32-bit hashes, half 20-bit values (many duplicates)
    _fill(keys, lambda s, e: torch.where(torch.arange(s, e, device="cuda") % 2 == 0,
                                         _hash(s, e, 3), _hash(s, e, 5) >> 12).to(torch.int32))
    ko = torch.empty_like(keys)
    po = torch.empty_like(keys)
    kt = torch.empty_like(keys)
    pt = torch.empty_like(keys)
    ops.radix_sort_u32(keys, bits_per_pass=8, keys_out=ko, perm_out=po, keys_tmp=kt, perm_tmp=pt)
    torch.cuda.synchronize()
    _check_sorted(keys, ko, po, "radix8")
    ko2 = torch.empty_like(keys)
    po2 = torch.empty_like(keys)
    for bits in (4, 1):  # the first sort's ping-pong buffers are free now
        announce("radix_sort_u32", bits, n)
        ops.radix_sort_u32(keys, bits_per_pass=bits, keys_out=ko2, perm_out=po2, keys_tmp=kt,
                           perm_tmp=pt)
        torch.cuda.synchronize()
        assert bool(torch.equal(po2, po)) and bool(torch.equal(ko2, ko)), f"radix{bits} differs"


def test_samplers_on_one_row_past_2p24(ops):
    """One row of 2^25 + 3 probabilities (weights), against the oracle."""
    length = (1 << 25) + 3
    announce("samplers on one row", length)
    probs = W.sample_probs(1, length, seed=25)
    theta = np.array([0.3125], np.float32)
    csum = np.cumsum(probs[0].astype(np.float64))
    g = int(to_host(ops.weighted_sample_f32(to_dev(probs), to_dev(theta)))[0])
    ref = int(oracle.weighted_sample_f32(probs, theta)[0])
    total = float(csum[-1])
    assert g == ref or draw_accept(g, csum, float(theta[0]) * total,
                                   draw_tol(float(theta[0]), total), length - 1), (g, ref)
    tok, cut = ops.topp_sample_f32(to_dev(probs), to_dev(theta), 0.9, with_cutoff=True)
    tok, cut = int(to_host(tok)[0]), int(to_host(cut)[0])
    rt, rc = oracle.topp_sample_f32(probs, theta, 0.9)
    if tok != int(rt[0]) or cut != int(rc[0]):
        sk, sp = oracle.sort_rows_f32(probs, descending=True)
        scs = np.cumsum(sk[0].astype(np.float64))
        assert topp_accept(cut, int(rc[0]), scs, 0.9), (cut, int(rc[0]))
        j = int(np.flatnonzero(sp[0] == tok)[0])
        ck = float(scs[cut])
        assert draw_accept(j, scs, float(theta[0]) * ck, draw_tol(float(theta[0]), ck), cut), \
            (tok, int(rt[0]))
    # exact case: weights 0 or 2^-24 (one in 16 set, so every running sum is
    # below 2^21 units and every threshold below 2^24 units), dyadic theta
    # and p: every fp32 sum and product is exact and the draws must be the
    # oracle's
    rng = np.random.default_rng(26)
    ex = ((rng.random((1, length)) < 1 / 16) * 2.0**-24).astype(np.float32)
    th = np.array([0.625], np.float32)
    assert float(ex.sum(dtype=np.float64)) < 2.0**-3
    assert int(to_host(ops.weighted_sample_f32(to_dev(ex), to_dev(th)))[0]) == \
        int(oracle.weighted_sample_f32(ex, th)[0])
    assert int(to_host(ops.topp_sample_f32(to_dev(ex), to_dev(th), 2.0**-4))[0]) == \
        int(oracle.topp_sample_f32(ex, th, 2.0**-4)[0][0])
