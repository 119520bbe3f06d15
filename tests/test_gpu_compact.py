"""GPU parity of Compress (mask compaction) and Split, through the C ABI.

Everything here is integer / bit-copy work, so it must match the oracle
exactly: kept values (compared as bit patterns), source indices, counts,
and the stable split permutation.
"""
import numpy as np
import pytest

import oracle
from gpu_util import announce, assert_equal_first_diff, to_dev, to_host
from paper_2505_15112_amd import workloads as W

pytestmark = pytest.mark.gpu

SIZES = [1, 5, 63, 64, 65, 255, 4095, 4096, 4097, 3 * 4096 + 5, 65_536, 3 * 32768 + 5,
         (1 << 20) + 17]


@pytest.fixture(scope="module")
def ops():
    from paper_2505_15112_amd import ops
    return ops


def _masks(n, seed):
    yield "bernoulli", W.mask_u8(n, seed=seed)
    yield "zeros", np.zeros(n, np.uint8)
    yield "ones", np.ones(n, np.uint8)
    yield "sparse", W.mask_u8(n, seed=seed, p_true=0.01)
    m = W.bytes_u8(n, seed=seed)  # arbitrary bytes: any non-zero byte counts as true
    yield "bytes", m


def _check_compact(ops, x, m, with_idx, what):
    out, idx, cnt = ops.compact_by_mask_f32(to_dev(x), to_dev(m), with_idx=with_idx)
    ref_out, ref_idx = oracle.compact_f32(x, m)
    c = int(to_host(cnt)[0])
    assert c == ref_out.size, f"{what}: count {c} != {ref_out.size}"
    assert_equal_first_diff(to_host(out)[:c].view(np.uint32), ref_out.view(np.uint32), what)
    if with_idx:
        assert_equal_first_diff(to_host(idx)[:c], ref_idx, what + " idx")


@pytest.mark.parametrize("n", SIZES)
def test_compact(ops, n):
    x = W.values_f32(n, seed=n)
    for name, m in _masks(n, n):
        announce("compact", n, name)
        _check_compact(ops, x, m, True, f"compact n={n} {name}")
    _check_compact(ops, x, W.mask_u8(n, seed=1), False, f"compact n={n} no idx")


@pytest.mark.parametrize("which", ["out", "idx"])
def test_compact_outputs_not_16_byte_aligned(ops, which):
    """Aligned input, an output 4 bytes off 16-byte alignment: the kept runs
    are written element by element instead of as aligned 16-byte quads."""
    import torch
    announce("compact unaligned output", which)
    n = 3 * 32768 + 5
    x = W.values_f32(n, seed=9)
    m = W.mask_u8(n, seed=9)
    ob = torch.empty(n + 1, dtype=torch.float32, device="cuda")
    ib = torch.empty(n + 1, dtype=torch.int32, device="cuda")
    out = ob[1:] if which == "out" else ob[:n]
    idx = ib[1:] if which == "idx" else ib[:n]
    out, idx, cnt = ops.compact_by_mask_f32(to_dev(x), to_dev(m), with_idx=True, out=out,
                                            idx_out=idx)
    ro, ri = oracle.compact_f32(x, m)
    c = int(cnt.item())
    assert c == ro.size
    assert_equal_first_diff(to_host(out)[:c].view(np.uint32), ro.view(np.uint32), which + " values")
    assert_equal_first_diff(to_host(idx)[:c], ri, which + " idx")


def test_compact_misaligned_and_empty(ops):
    import torch
    announce("compact misaligned/empty")
    n = 10_007
    x = W.values_f32(n + 1, seed=3)
    m = W.mask_u8(n + 1, seed=3)
    out, idx, cnt = ops.compact_by_mask_f32(to_dev(x)[1:], to_dev(m)[1:], with_idx=True)
    ro, ri = oracle.compact_f32(x[1:], m[1:])
    c = int(cnt.item())
    assert c == ro.size
    assert_equal_first_diff(to_host(out)[:c].view(np.uint32), ro.view(np.uint32), "misaligned")
    assert_equal_first_diff(to_host(idx)[:c], ri, "misaligned idx")
    e = torch.empty(0, dtype=torch.float32, device="cuda")
    _, _, c0 = ops.compact_by_mask_f32(e, torch.empty(0, dtype=torch.uint8, device="cuda"))
    assert int(c0.item()) == 0


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_compact_config_n2_28(ops, seed):
    announce("compact config n=2^28", seed)
    n = 1 << 28
    x = W.values_f32(n, seed=seed)
    m = W.mask_u8(n, seed=seed)
    _check_compact(ops, x, m, True, f"compact config seed={seed}")


def _check_split(ops, k, f, idx_in, what):
    ki = k.view(np.int32)
    ko, io, nt = ops.split_by_flags_u32(to_dev(ki), to_dev(f),
                                        idx_in=None if idx_in is None else to_dev(idx_in))
    rk, ri, rn = oracle.split_u32(k, f, idx_in=idx_in)
    assert int(to_host(nt)[0]) == rn, what
    assert_equal_first_diff(to_host(ko).view(np.uint32), rk, what + " keys")
    assert_equal_first_diff(to_host(io), ri, what + " idx")


@pytest.mark.parametrize("n", SIZES)
def test_split(ops, n):
    k = W.keys_u32(n, seed=n)
    for name, f in _masks(n, n + 1):
        announce("split", n, name)
        _check_split(ops, k, f, None, f"split n={n} {name}")
    perm = np.random.default_rng(n).permutation(n).astype(np.int32)
    _check_split(ops, k, W.mask_u8(n, seed=2), perm, f"split n={n} idx_in")


def test_split_misaligned(ops):
    """Keys and flags one element off alignment: the element-wise tile path."""
    n = 3 * 32768 + 5
    announce("split misaligned", n)
    k = W.keys_u32(n + 1, seed=31)
    f = W.mask_u8(n + 1, seed=32)
    kd, fd = to_dev(k.view(np.int32)), to_dev(f)
    ko, io, nt = ops.split_by_flags_u32(kd[1:], fd[1:])
    rk, ri, rn = oracle.split_u32(k[1:], f[1:])
    assert int(nt.item()) == rn
    assert_equal_first_diff(to_host(ko).view(np.uint32), rk, "split misaligned keys")
    assert_equal_first_diff(to_host(io), ri, "split misaligned idx")


def test_split_repeated_calls_share_workspace(ops):
    """One workspace across many calls and sizes: the epoch-tagged flag count
    must never leak from one call into the next."""
    announce("split shared ws")
    ws = ops.workspace(4, "cuda", 1 << 20)
    for i, n in enumerate([1 << 20, 1000, 4097, 1 << 20, 7, 65_536]):
        k = W.keys_u32(n, seed=i)
        f = W.mask_u8(n, seed=i, p_true=0.3 if i % 2 else 0.7)
        ko, io, nt = ops.split_by_flags_u32(to_dev(k.view(np.int32)), to_dev(f), ws=ws)
        rk, ri, rn = oracle.split_u32(k, f)
        assert int(nt.item()) == rn, (i, n)
        assert_equal_first_diff(to_host(io), ri, f"shared ws call {i}")
        x = W.values_f32(n, seed=i)
        out, idx, cnt = ops.compact_by_mask_f32(to_dev(x), to_dev(f), with_idx=True, ws=ws)
        ro, rio = oracle.compact_f32(x, f)
        assert int(cnt.item()) == ro.size
        assert_equal_first_diff(to_host(idx)[: ro.size], rio, f"shared ws compact {i}")
