"""libscan.so on the CPU: it loads without a GPU, exports every function that
include/libscan.h declares, and rejects bad arguments before any HIP call.

No call here reaches a kernel launch: every call made with fake device
addresses fails validation first, by construction of its arguments.
"""
import ctypes
import os

import pytest

from paper_2505_15112_amd import _lib

if not (os.path.exists(_lib.LIB_PATH) and os.path.exists(_lib.LIB_ADV_PATH)):
    # load what is built; build only if nothing is
    from paper_2505_15112_amd import build as _build
    _build.build()

P = ctypes.c_void_p
X = P(0x100000)      # fake, never dereferenced
Y = P(0x900000)
WS = P(0x4000000)
XB = P(1 << 40)      # far apart, for large fake sizes
YB = P(1 << 41)
BIG = 1 << 30


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def test_every_declared_symbol_is_exported(lib):
    declared = _lib.header_functions()
    assert len(declared) >= 16
    for name in declared:
        assert hasattr(lib, name), name
        assert name in _lib.SIGNATURES, f"{name} missing from the binding"
    assert sorted(_lib.SIGNATURES) == declared


def test_adversarial_build_exports_the_same_symbols_and_checks(lib):
    """libscan_adv.so (the test build with pauses) loads beside libscan.so,
    exports the same entry points and validates the same way."""
    adv = _lib.load_adversarial()
    assert adv is not lib
    for name in _lib.header_functions():
        assert hasattr(adv, name), name
    assert adv.scan_inclusive_i32(X, Y, -1, WS, BIG, None) == _lib.EINVAL
    assert adv.scan_inclusive_i32(X, Y, 1 << 20, WS, 8, None) == _lib.ENOSPACE


def test_version_and_strings(lib):
    assert lib.libscan_version() >= 100
    for st in (0, -1, -2, -3, -4, 7):
        assert isinstance(lib.libscan_status_string(st), bytes)
    assert lib.libscan_status_string(-2) == b"workspace too small"


def test_workspace_bytes(lib):
    out = ctypes.c_size_t(0)
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN, 0, 0, 0, 0, ctypes.byref(out)) == 0
    small = out.value
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN, 1 << 28, 0, 0, 0, ctypes.byref(out)) == 0
    assert out.value >= small + 8 * ((1 << 28) // 16384)
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN_RSS, 1 << 20, 0, 0, 0, ctypes.byref(out)) == 0
    assert lib.libscan_workspace_bytes(99, 10, 0, 0, 0, ctypes.byref(out)) == _lib.EINVAL
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN, -1, 0, 0, 0, ctypes.byref(out)) == _lib.EINVAL
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN, 10, 0, 0, 0, None) == _lib.EINVAL
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN, 1 << 40, 0, 0, 0,
                                       ctypes.byref(out)) == _lib.ERANGE


SCANS = ["scan_inclusive_i32", "scan_exclusive_i32", "scan_inclusive_f32", "scan_exclusive_f32",
         "scan_inclusive_f16f32", "scan_exclusive_f16f32", "scan_inclusive_f16f32_mfma",
         "scan_inclusive_f16f32_wave", "scan_inclusive_rss_i32",
         "scan_inclusive_rss_f32"]


@pytest.mark.parametrize("name", SCANS)
def test_scan_validation(lib, name):
    fn = getattr(lib, name)
    assert fn(X, Y, -1, WS, BIG, None) == _lib.EINVAL           # negative size
    assert fn(None, Y, 10, WS, BIG, None) == _lib.EINVAL        # NULL input
    assert fn(X, None, 10, WS, BIG, None) == _lib.EINVAL        # NULL output
    assert fn(X, P(0x100004), 100, WS, BIG, None) == _lib.EINVAL  # partial overlap
    assert fn(X, Y, 1 << 40, WS, BIG, None) == _lib.ERANGE      # too long
    assert fn(X, Y, 1 << 20, WS, 8, None) == _lib.ENOSPACE      # workspace too small
    assert fn(X, Y, 1 << 20, P(0x4000004), BIG, None) == _lib.EINVAL  # misaligned workspace
    assert fn(X, Y, 1 << 20, None, BIG, None) == _lib.EINVAL    # NULL workspace
    assert fn(None, None, 0, None, 0, None) == _lib.OK          # empty: nothing to do


def test_mixed_type_scans_reject_any_overlap(lib):
    # fp16 in / fp32 out may not alias at all, not even exactly
    assert lib.scan_inclusive_f16f32(X, X, 100, WS, BIG, None) == _lib.EINVAL
    assert lib.scan_inclusive_f16f32_mfma(X, X, 100, WS, BIG, None) == _lib.EINVAL
    assert lib.scan_inclusive_f16f32_wave(X, X, 100, WS, BIG, None) == _lib.EINVAL
    # the matrix-core scan needs a 16-byte aligned input
    assert lib.scan_inclusive_f16f32_mfma(P(0x100002), Y, 100, WS, BIG, None) == _lib.EINVAL
    assert lib.scan_exclusive_u8i32(X, X, 100, None, WS, BIG, None) == _lib.EINVAL
    for name in ("scan_exclusive_u8i32_mfma", "scan_exclusive_u8i32_wave"):
        fn = getattr(lib, name)
        assert fn(X, X, 100, None, WS, BIG, None) == _lib.EINVAL        # overlap
        assert fn(X, Y, -1, None, WS, BIG, None) == _lib.EINVAL         # negative size
        assert fn(None, Y, 10, None, WS, BIG, None) == _lib.EINVAL      # NULL input
        assert fn(X, Y, 1 << 40, None, WS, BIG, None) == _lib.ERANGE    # too long
        assert fn(X, Y, 1 << 20, None, WS, 8, None) == _lib.ENOSPACE    # workspace too small
        assert fn(None, None, 0, None, None, 0, None) == _lib.OK        # empty
    # the matrix-core byte scan needs a 16-byte aligned input
    assert lib.scan_exclusive_u8i32_mfma(P(0x100001), Y, 100, None, WS, BIG, None) == _lib.EINVAL


def test_carry_validation(lib):
    for name in ("scan_inclusive_i32_carry", "scan_exclusive_i32_carry",
                 "scan_inclusive_f32_carry", "scan_exclusive_f32_carry"):
        fn = getattr(lib, name)
        assert fn(X, Y, -5, None, None, WS, BIG, None) == _lib.EINVAL
        # total written inside the output range
        assert fn(X, Y, 100, None, P(0x900008), WS, BIG, None) == _lib.EINVAL
        assert fn(X, Y, 1 << 20, None, None, WS, 16, None) == _lib.ENOSPACE


def test_python_binding_needs_gpu_tensors():
    import torch
    from paper_2505_15112_amd import ops
    with pytest.raises(ValueError):
        ops.scan_inclusive_i32(torch.zeros(10, dtype=torch.int32))
    with pytest.raises(TypeError):
        ops.scan_inclusive_i32(torch.zeros(10, dtype=torch.int64))


def test_rows_validation(lib):
    for name in ("scan_rows_i32", "scan_rows_f32"):
        fn = getattr(lib, name)
        assert fn(X, Y, -1, 10, 0, WS, BIG, None) == _lib.EINVAL
        assert fn(X, Y, 10, -1, 0, WS, BIG, None) == _lib.EINVAL
        assert fn(None, Y, 10, 10, 0, WS, BIG, None) == _lib.EINVAL
        assert fn(X, P(0x100010), 10, 10, 0, WS, BIG, None) == _lib.EINVAL  # overlap
        assert fn(X, Y, 1 << 20, 1 << 20, 0, WS, BIG, None) == _lib.ERANGE
        assert fn(X, Y, 1 << 24, 8192, 0, WS, BIG, None) == _lib.ERANGE      # grid too large
        assert fn(XB, YB, 100, 100_000, 0, WS, 64, None) == _lib.ENOSPACE
        assert fn(None, None, 0, 10, 0, None, 0, None) == _lib.OK


def test_topp_validation(lib):
    fn = lib.topp_cutoff_f32
    assert fn(X, Y, 4, 10, float("nan"), WS, BIG, None) == _lib.EINVAL
    assert fn(X, None, 4, 10, 0.9, WS, BIG, None) == _lib.EINVAL
    assert fn(None, Y, 4, 10, 0.9, WS, BIG, None) == _lib.EINVAL
    assert fn(X, P(0x100008), 4, 10, 0.9, WS, BIG, None) == _lib.EINVAL  # cutoff inside probs
    assert fn(X, Y, 1, 1 << 31, 0.9, WS, BIG, None) == _lib.ERANGE
    assert fn(XB, YB, 128, 131072, 0.9, WS, 256, None) == _lib.ENOSPACE
    assert fn(None, None, 0, 10, 0.9, None, 0, None) == _lib.OK


def test_rows_workspace_bytes(lib):
    out = ctypes.c_size_t(0)
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN_ROWS, 0, 128, 131072, 0,
                                       ctypes.byref(out)) == 0
    assert out.value >= 256 + 128 * 4 * 8
    assert lib.libscan_workspace_bytes(_lib.OP_SCAN_ROWS, 0, 1000, 100, 0, ctypes.byref(out)) == 0
    assert out.value == 256  # one wavefront per row needs no status words


def test_compact_validation(lib):
    fn = lib.compact_by_mask_f32
    C = P(0x7000000)
    assert fn(X, Y, WS, None, C, -1, WS, BIG, None) == _lib.EINVAL
    assert fn(X, Y, P(0x2000000), None, None, 10, WS, BIG, None) == _lib.EINVAL   # no count
    assert fn(None, Y, P(0x2000000), None, C, 10, WS, BIG, None) == _lib.EINVAL
    assert fn(X, Y, P(0x100010), None, C, 10, WS, BIG, None) == _lib.EINVAL     # out over x
    assert fn(X, Y, P(0x2000000), P(0x2000010), C, 10, WS, BIG, None) == _lib.EINVAL  # idx/out
    assert fn(XB, YB, P(1 << 42), None, C, 1 << 31, WS, BIG, None) == _lib.ERANGE
    assert fn(XB, YB, P(1 << 42), None, C, 1 << 20, WS, 64, None) == _lib.ENOSPACE


def test_split_validation(lib):
    fn = lib.split_by_flags_u32
    KO, IO, NT = P(0x2000000), P(0x3000000), P(0x7000000)
    assert fn(X, None, Y, KO, IO, NT, -1, WS, BIG, None) == _lib.EINVAL
    assert fn(None, None, Y, KO, IO, NT, 10, WS, BIG, None) == _lib.EINVAL
    assert fn(X, None, None, KO, IO, NT, 10, WS, BIG, None) == _lib.EINVAL      # no flags
    assert fn(X, None, Y, X, IO, NT, 10, WS, BIG, None) == _lib.EINVAL         # in place
    assert fn(X, None, Y, KO, P(0x2000004), NT, 10, WS, BIG, None) == _lib.EINVAL
    assert fn(X, IO, Y, KO, IO, NT, 10, WS, BIG, None) == _lib.EINVAL          # idx_out == idx_in
    assert fn(XB, None, YB, P(1 << 42), None, None, 1 << 31, WS, BIG, None) == _lib.ERANGE
    assert fn(XB, None, YB, P(1 << 42), None, None, 1 << 20, WS, 64, None) == _lib.ENOSPACE
    assert fn(None, None, None, None, None, None, 0, None, 0, None) == _lib.OK


@pytest.mark.parametrize("name,elem", [("radix_sort_i32", 4), ("radix_sort_f32", 4),
                                       ("radix_sort_f16", 2)])
def test_typed_radix_validation(lib, name, elem):
    fn = getattr(lib, name)
    KO, PO, KT, PT = P(0x2000000), P(0x3000000), P(0x4000000), P(0x5000000)
    W2 = P(0x60000000)
    assert fn(X, KO, PO, KT, PT, -1, 0, W2, BIG, None) == _lib.EINVAL
    assert fn(X, KO, PO, None, PT, 10, 0, W2, BIG, None) == _lib.EINVAL      # no keys_tmp
    assert fn(X, KO, PO, KT, None, 10, 1, W2, BIG, None) == _lib.EINVAL      # perm without tmp
    assert fn(X, X, PO, KT, PT, 10, 0, W2, BIG, None) == _lib.EINVAL         # in place
    # keys_tmp overlapping keys_out by one element
    assert fn(X, KO, PO, P(0x2000000 + 9 * elem), PT, 10, 0, W2, BIG, None) == _lib.EINVAL
    assert fn(XB, YB, None, P(1 << 42), None, 1 << 31, 0, W2, BIG, None) == _lib.ERANGE
    assert fn(X, KO, PO, KT, PT, 1000, 0, W2, 64, None) == _lib.ENOSPACE
    assert fn(None, None, None, None, None, 0, 1, None, 0, None) == _lib.OK


def test_radix_validation(lib):
    fn = lib.radix_sort_u32
    KO, PO, KT, PT = P(0x2000000), P(0x3000000), P(0x4000000), P(0x5000000)
    W2 = P(0x60000000)
    assert fn(X, KO, PO, KT, PT, -1, 4, W2, BIG, None) == _lib.EINVAL
    assert fn(X, KO, PO, KT, PT, 10, 2, W2, BIG, None) == _lib.EINVAL        # bits not 1/4/8
    assert fn(X, KO, PO, KT, PT, 10, 16, W2, BIG, None) == _lib.EINVAL
    assert fn(X, KO, PO, None, PT, 10, 4, W2, BIG, None) == _lib.EINVAL      # no keys_tmp
    assert fn(X, KO, PO, KT, None, 10, 4, W2, BIG, None) == _lib.EINVAL      # perm without tmp
    assert fn(X, X, PO, KT, PT, 10, 4, W2, BIG, None) == _lib.EINVAL         # in place
    assert fn(X, KO, PO, P(0x2000008), PT, 10, 4, W2, BIG, None) == _lib.EINVAL
    assert fn(XB, YB, None, P(1 << 42), None, 1 << 31, 4, W2, BIG, None) == _lib.ERANGE
    assert fn(X, KO, PO, KT, PT, 1000, 4, W2, 64, None) == _lib.ENOSPACE
    assert fn(None, None, None, None, None, 0, 4, None, 0, None) == _lib.OK
    out = ctypes.c_size_t(0)
    assert lib.libscan_workspace_bytes(_lib.OP_RADIX_SORT, 1 << 26, 0, 0, 4, ctypes.byref(out)) == 0
    assert out.value >= 256 + 16 * 4 * ((1 << 26) // 8192)
    assert lib.libscan_workspace_bytes(_lib.OP_RADIX_SORT, 1 << 26, 0, 0, 8, ctypes.byref(out)) == 0
    assert out.value >= 256 + 256 * 4 * ((1 << 26) // 8192)
    assert lib.libscan_workspace_bytes(_lib.OP_RADIX_SORT, 100, 0, 0, 3, ctypes.byref(out)) == _lib.EINVAL


def test_sort_rows_validation(lib):
    fn = lib.radix_sort_rows_f32
    KO, PO, KT, PT = P(0x2000000), P(0x3000000), P(0x4000000), P(0x5000000)
    W2 = P(0x60000000)
    assert fn(X, KO, PO, KT, PT, -1, 10, 0, W2, BIG, None) == _lib.EINVAL
    assert fn(X, KO, PO, KT, PT, 10, -1, 0, W2, BIG, None) == _lib.EINVAL
    assert fn(X, KO, PO, None, PT, 4, 10, 0, W2, BIG, None) == _lib.EINVAL     # no keys_tmp
    assert fn(X, KO, PO, KT, None, 4, 10, 1, W2, BIG, None) == _lib.EINVAL     # perm without tmp
    assert fn(X, X, PO, KT, PT, 4, 10, 0, W2, BIG, None) == _lib.EINVAL        # in place
    assert fn(X, KO, PO, P(0x2000000 + 39 * 4), PT, 4, 10, 0, W2, BIG, None) == _lib.EINVAL
    assert fn(XB, YB, None, P(1 << 42), None, 1 << 16, 1 << 15, 0, W2, BIG,
              None) == _lib.ERANGE                                              # > INT32_MAX keys
    assert fn(XB, YB, None, P(1 << 42), None, (1 << 24) + 1, 8, 0, W2, BIG,
              None) == _lib.ERANGE                                              # grid too large
    assert fn(X, KO, PO, KT, PT, 16, 10000, 0, W2, 64, None) == _lib.ENOSPACE
    assert fn(None, None, None, None, None, 0, 10, 0, None, 0, None) == _lib.OK
    assert fn(None, None, None, None, None, 10, 0, 0, None, 0, None) == _lib.OK
    out = ctypes.c_size_t(0)
    assert lib.libscan_workspace_bytes(_lib.OP_SORT_ROWS, 0, 64, 1 << 17, 0,
                                       ctypes.byref(out)) == _lib.OK
    assert out.value >= 256 + 64 * 256 * 4 * ((1 << 17) // 8192)


def test_weighted_sample_validation(lib):
    fn = lib.weighted_sample_f32
    TH, OUT = P(0x2000000), P(0x3000000)
    assert fn(X, TH, OUT, -1, 10, WS, BIG, None) == _lib.EINVAL
    assert fn(None, TH, OUT, 4, 10, WS, BIG, None) == _lib.EINVAL
    assert fn(X, None, OUT, 4, 10, WS, BIG, None) == _lib.EINVAL               # no theta
    assert fn(X, TH, None, 4, 10, WS, BIG, None) == _lib.EINVAL
    assert fn(X, TH, P(0x100008), 4, 10, WS, BIG, None) == _lib.EINVAL         # out inside w
    assert fn(X, TH, P(0x2000004), 4, 10, WS, BIG, None) == _lib.EINVAL        # out over theta
    assert fn(XB, TH, OUT, 1, 1 << 31, WS, BIG, None) == _lib.ERANGE
    assert fn(XB, TH, OUT, 128, 131072, WS, 256, None) == _lib.ENOSPACE
    assert fn(None, None, None, 0, 10, None, 0, None) == _lib.OK
    out = ctypes.c_size_t(0)
    # every length needs the per-tile sums and the per-row arrival counters
    assert lib.libscan_workspace_bytes(_lib.OP_WEIGHTED_SAMPLE, 0, 1000, 100, 0,
                                       ctypes.byref(out)) == _lib.OK
    assert out.value >= 256 + 1000 * 16


def test_topp_sample_validation(lib):
    fn = lib.topp_sample_f32
    TH, TOK, CUT = P(0x2000000), P(0x3000000), P(0x3100000)
    SC, W2 = P(0x40000000), P(0x60000000)
    assert fn(X, TH, float("nan"), TOK, CUT, 4, 10, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, None, 0.9, TOK, CUT, 4, 10, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, TH, 0.9, None, CUT, 4, 10, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, TH, 0.9, TOK, TOK, 4, 10, SC, BIG, W2, BIG, None) == _lib.EINVAL  # cutoff == token
    assert fn(X, TH, 0.9, TOK, P(0x100004), 4, 10, SC, BIG, W2, BIG, None) == _lib.EINVAL
    # scratch: required, aligned, large enough, and clear of inputs, outputs and the workspace
    assert fn(X, TH, 0.9, TOK, CUT, 4, 10, None, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, TH, 0.9, TOK, CUT, 4, 10, P(0x40000004), BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, TH, 0.9, TOK, CUT, 4, 10, SC, 64, W2, BIG, None) == _lib.ENOSPACE
    assert fn(X, TH, 0.9, TOK, CUT, 4, 10, P(0x3000000 - 256), 1024, W2, BIG, None) == _lib.EINVAL
    assert fn(X, TH, 0.9, TOK, CUT, 4, 10, SC, 1 << 20, P(0x40000100), 1 << 20,
              None) == _lib.EINVAL
    assert fn(X, TH, 0.9, TOK, CUT, 4, 10, SC, BIG, W2, 64, None) == _lib.ENOSPACE
    assert fn(XB, TH, 0.9, TOK, CUT, 1 << 16, 1 << 15, SC, BIG, W2, BIG, None) == _lib.ERANGE
    assert fn(None, None, 0.9, None, None, 0, 10, None, 0, None, 0, None) == _lib.OK
    out = ctypes.c_size_t(0)
    assert lib.libscan_workspace_bytes(_lib.OP_TOPP_SAMPLE, 0, 64, 1 << 17, 0,
                                       ctypes.byref(out)) == _lib.OK
    assert out.value >= 256 + 64 * 256 * 4 * ((1 << 17) // 8192)
    assert lib.libscan_scratch_bytes(_lib.OP_TOPP_SAMPLE, 64, 1 << 17, 0,
                                     ctypes.byref(out)) == _lib.OK
    assert out.value >= 16 * 64 * (1 << 17)
    assert lib.libscan_scratch_bytes(_lib.OP_TOPP_SAMPLE, 1 << 16, 1 << 15, 0,
                                     ctypes.byref(out)) == _lib.ERANGE
    assert lib.libscan_scratch_bytes(_lib.OP_SCAN, 4, 10, 0, ctypes.byref(out)) == _lib.EINVAL
    assert lib.libscan_scratch_bytes(_lib.OP_TOPP_SAMPLE, 4, 10, 0, None) == _lib.EINVAL


def test_topk_validation(lib):
    fn = lib.topk_rows_f32
    VO, IO, SC, W2 = P(0x2000000), P(0x3000000), P(0x40000000), P(0x60000000)
    assert fn(X, VO, IO, -1, 10, 3, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, VO, IO, 4, 10, 11, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL   # k > len
    assert fn(X, VO, IO, 4, 10, -1, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(None, VO, IO, 4, 10, 3, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, VO, None, 4, 10, 3, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, P(0x100010), IO, 4, 10, 3, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL  # over x
    assert fn(X, VO, P(0x2000008), 4, 10, 3, 1, SC, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, VO, IO, 4, 10, 3, 1, None, BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, VO, IO, 4, 10, 3, 1, P(0x40000008), BIG, W2, BIG, None) == _lib.EINVAL
    assert fn(X, VO, IO, 4, 10, 3, 1, SC, 16, W2, BIG, None) == _lib.ENOSPACE
    assert fn(X, VO, IO, 4, 10, 3, 1, SC, 1 << 20, P(0x40000100), 1 << 20, None) == _lib.EINVAL
    assert fn(X, VO, IO, 4, 10, 3, 1, SC, BIG, W2, 64, None) == _lib.ENOSPACE
    assert fn(XB, VO, IO, 1, 1 << 31, 3, 1, SC, BIG, W2, BIG, None) == _lib.ERANGE
    assert fn(XB, VO, IO, 1 << 16, 1 << 16, 1 << 15, 1, SC, BIG, W2, BIG, None) == _lib.ERANGE
    assert fn(None, None, None, 0, 10, 3, 1, None, 0, None, 0, None) == _lib.OK
    assert fn(None, None, None, 4, 10, 0, 1, None, 0, None, 0, None) == _lib.OK    # k = 0
    out = ctypes.c_size_t(0)
    assert lib.libscan_workspace_bytes(_lib.OP_TOPK, 4096, 128, 131072, 0,
                                       ctypes.byref(out)) == _lib.OK
    assert out.value >= 256 + 128 * 4 * (16 + 256 * 4)
    assert lib.libscan_workspace_bytes(_lib.OP_TOPK, 11, 4, 10, 0, ctypes.byref(out)) == _lib.EINVAL
    assert lib.libscan_scratch_bytes(_lib.OP_TOPK, 128, 131072, 4096, ctypes.byref(out)) == _lib.OK
    assert out.value >= 8 * 128 * 4096            # the kept values and indices
    assert lib.libscan_scratch_bytes(_lib.OP_TOPK, 4, 131072, 9000, ctypes.byref(out)) == _lib.OK
    assert out.value >= 16 * 4 * 9000             # and the row sort's ping-pong buffers
    # k <= 256: 1024 candidate slots (keys and indices) per tile of the row
    assert lib.libscan_scratch_bytes(_lib.OP_TOPK, 128, 131072, 64, ctypes.byref(out)) == _lib.OK
    assert out.value >= 128 * 16 * 8192           # 8192-element tiles
    assert lib.libscan_scratch_bytes(_lib.OP_TOPK, 3, 16384, 256, ctypes.byref(out)) == _lib.OK
    assert out.value >= 3 * 4 * 8192              # 4096-element tiles up to 16384


def test_workspace_error_validation(lib):
    """libscan_workspace_error checks its arguments before enqueueing anything."""
    E = P(0x200000)
    assert lib.libscan_workspace_error(None, 4096, E, 1, None) == _lib.EINVAL
    assert lib.libscan_workspace_error(P(0x4000008), 4096, E, 1, None) == _lib.EINVAL  # alignment
    assert lib.libscan_workspace_error(WS, 4096, None, 1, None) == _lib.EINVAL
    assert lib.libscan_workspace_error(WS, 4096, P(0x200002), 1, None) == _lib.EINVAL
    assert lib.libscan_workspace_error(WS, 255, E, 1, None) == _lib.ENOSPACE
    assert lib.libscan_workspace_error(WS, 4096, P(0x4000000 + 12), 1, None) == _lib.EINVAL


def test_noalloc_validation(lib):
    """The entry point without a workspace: sizes beyond its static array are
    rejected before any HIP call, as are negative sizes, NULL data and a
    partial overlap."""
    f = lib.scan_inclusive_i32_noalloc
    assert f(X, Y, -1, None) == _lib.EINVAL
    assert f(None, Y, 5, None) == _lib.EINVAL
    assert f(X, None, 5, None) == _lib.EINVAL
    assert f(X, P(0x100000 + 4), 5, None) == _lib.EINVAL
    assert f(XB, YB, (1 << 31) + 1, None) == _lib.ERANGE
    assert f(XB, YB, 1 << 40, None) == _lib.ERANGE
    assert f(None, None, 0, None) == _lib.OK


def _gpu_present():
    import torch
    return os.path.exists("/dev/kfd") or torch.cuda.device_count() > 0


@pytest.mark.skipif(_gpu_present(), reason="needs a box without a GPU: the calls below launch "
                    "kernels on fake addresses")
def test_well_formed_calls_without_a_gpu_return_ehip(lib):
    """Calls that pass validation reach the HIP launch, which fails on a box
    without a GPU: the status is LIBSCAN_EHIP, not a crash or a hang."""
    ws_bytes = 1 << 20
    assert lib.scan_inclusive_i32(X, Y, 1000, WS, ws_bytes, None) == _lib.EHIP
    assert lib.scan_exclusive_f32(X, Y, 100_000, WS, ws_bytes, None) == _lib.EHIP
    assert lib.libscan_workspace_init(WS, ws_bytes, None) == _lib.EHIP
    assert lib.libscan_workspace_error(WS, ws_bytes, P(0x200000), 1, None) == _lib.EHIP
    assert lib.scan_inclusive_i32_noalloc(X, Y, 1000, None) == _lib.EHIP
