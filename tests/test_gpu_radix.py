"""GPU parity of the LSD radix sort (1, 4 and 8 bits per pass), through the C ABI.

A stable sort has exactly one correct output, so keys and permutation must
equal the oracle's bit for bit, and the pass widths must agree.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, assert_equal_first_diff, to_dev, to_host
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu

SIZES = [1, 2, 5, 63, 64, 65, 255, 4095, 4096, 4097, 3 * 4096 + 5, 8191, 8192, 8193, 65_539,
         (1 << 20) + 17]


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


def _keysets(n, seed):
    yield "uniform", W.keys_u32(n, seed=seed)
    yield "mod16", W.keys_u32(n, seed=seed) % np.uint32(16)       # heavy ties: stability
    yield "equal", np.full(n, 0xDEADBEEF, np.uint32)
    yield "descending", np.arange(n, 0, -1, dtype=np.int64).astype(np.uint32) * np.uint32(4099)
    yield "high_bit", (W.keys_u32(n, seed=seed) | np.uint32(0x80000000)) ^ np.uint32(
        (np.arange(n) % 2) << 31)
    # one byte varies, the others fixed: 255 empty digits per pass but one
    yield "one_byte", (W.keys_u32(n, seed=seed) & np.uint32(0x00FF0000)) | np.uint32(0x12003456)


def _check(ops, keys, bits, with_perm, what):
    ko, po = ops.radix_sort_u32(to_dev(keys.view(np.int32)), bits_per_pass=bits,
                                with_perm=with_perm)
    rk, rp = oracle.sort_u32(keys)
    assert_equal_first_diff(to_host(ko).view(np.uint32), rk, what + " keys")
    if with_perm:
        assert_equal_first_diff(to_host(po), rp, what + " perm")


@pytest.mark.parametrize("n", SIZES)
@pytest.mark.parametrize("bits", [8, 4, 1])
def test_radix(ops, n, bits):
    for name, k in _keysets(n, n):
        announce("radix", n, bits, name)
        _check(ops, k, bits, True, f"radix{bits} n={n} {name}")
    _check(ops, W.keys_u32(n, seed=7), bits, False, f"radix{bits} n={n} keys only")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_radix_config_n2_26(ops, seed):
    announce("radix config n=2^26", seed)
    n = 1 << 26
    keys = W.keys_u32(n, seed=seed)
    rk, rp = oracle.sort_u32(keys)
    outs = {}
    for bits in (8, 4, 1):
        ko, po = ops.radix_sort_u32(to_dev(keys.view(np.int32)), bits_per_pass=bits)
        outs[bits] = (to_host(ko).view(np.uint32), to_host(po))
        assert_equal_first_diff(outs[bits][0], rk, f"config radix{bits} keys")
        assert_equal_first_diff(outs[bits][1], rp, f"config radix{bits} perm")
    assert np.array_equal(outs[1][1], outs[4][1]) and np.array_equal(outs[8][1], outs[4][1])
