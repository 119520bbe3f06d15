"""The CPU oracle against its pins (see oracle_pins.py).  CPU only."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import oracle_pins as P


@pytest.mark.parametrize("check", P.ALL_CHECKS, ids=lambda f: f.__name__)
def test_pin(check):
    check(oracle.default())


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(-2**31, 2**31 - 1), max_size=300))
def test_scan_i32_property(xs):
    x = np.array(xs, np.int32)
    got = oracle.scan_i32(x)
    want = [P._wrap(sum(xs[: i + 1])) for i in range(len(xs))]
    assert got.tolist() == want


@settings(max_examples=40, deadline=None)
@given(st.lists(st.integers(0, 255), max_size=300))
def test_scan_u8_property(xs):
    y, t = oracle.scan_u8(np.array(xs, np.uint8))
    assert y.tolist() == [sum(xs[:i]) for i in range(len(xs))]
    assert t == sum(xs)


def test_empty_inputs():
    o = oracle.default()
    e32 = np.zeros(0, np.int32)
    assert o.scan_i32(e32).size == 0 and o.scan_i32(e32, exclusive=True).size == 0
    y, a = o.scan_f32(np.zeros(0, np.float32))
    assert y.size == 0 and a.size == 0
    y, t = o.scan_u8(np.zeros(0, np.uint8))
    assert y.size == 0 and t == 0
    out, idx = o.compact_f32(np.zeros(0, np.float32), np.zeros(0, np.uint8))
    assert out.size == 0 and idx.size == 0
    ko, io, nt = o.split_u32(np.zeros(0, np.uint32), np.zeros(0, np.uint8))
    assert ko.size == 0 and nt == 0
    ko, perm = o.sort_u32(np.zeros(0, np.uint32))
    assert ko.size == 0 and perm.size == 0
