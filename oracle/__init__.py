"""Serial CPU oracle for the scan hot path (numpy front end over liboracle.so).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this package.  The product path
(``paper_2505_15112_amd``) never imports it and shares no code with it.

Every function is the plain definition of an operation of "Parallel Scan on
Ascend AI Accelerators", implemented in ``oracle.c`` as one serial loop:
integers wrap modulo 2^32, floating-point sums accumulate in float64.

``Oracle(path)`` binds the same front end to another build of ``oracle.c``;
the pin tests use that to check that deliberately broken builds fail them.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_i64 = ctypes.c_int64
_p = ctypes.c_void_p

_SIGNATURES = {
    "oracle_scan_inclusive_i32": ([_p, _p, _i64], None),
    "oracle_scan_exclusive_i32": ([_p, _p, _i64], None),
    "oracle_scan_inclusive_f32": ([_p, _p, _p, _i64], None),
    "oracle_scan_exclusive_f32": ([_p, _p, _p, _i64], None),
    "oracle_scan_inclusive_f16": ([_p, _p, _p, _i64], None),
    "oracle_scan_exclusive_f16": ([_p, _p, _p, _i64], None),
    "oracle_scan_exclusive_u8": ([_p, _p, _i64, _p], None),
    "oracle_scan_inclusive_u8": ([_p, _p, _i64], None),
    "oracle_scan_rows_i32": ([_p, _p, _i64, _i64, ctypes.c_int], None),
    "oracle_scan_rows_f32": ([_p, _p, _p, _i64, _i64, ctypes.c_int], None),
    "oracle_compact_f32": ([_p, _p, _p, _p, _i64], _i64),
    "oracle_split_u32": ([_p, _p, _p, _p, _p, _i64], _i64),
    "oracle_sort_u32": ([_p, _p, _p, _i64], ctypes.c_int),
    "oracle_sort_i32": ([_p, _p, _p, _i64, ctypes.c_int], ctypes.c_int),
    "oracle_sort_f32": ([_p, _p, _p, _i64, ctypes.c_int], ctypes.c_int),
    "oracle_sort_f16": ([_p, _p, _p, _i64, ctypes.c_int], ctypes.c_int),
    "oracle_sort_rows_f32": ([_p, _p, _p, _i64, _i64, ctypes.c_int], ctypes.c_int),
    "oracle_weighted_sample_f32": ([_p, _p, _p, _i64, _i64], None),
    "oracle_topp_sample_f32": ([_p, _p, ctypes.c_float, _p, _p, _i64, _i64], ctypes.c_int),
    "oracle_topk_rows_f32": ([_p, _p, _p, _i64, _i64, _i64, ctypes.c_int], ctypes.c_int),
    "oracle_topp_cutoff_f32": ([_p, _p, _i64, _i64, ctypes.c_float], None),
    "oracle_half_to_double": ([ctypes.c_uint16], ctypes.c_double),
}


def _ptr(a):
    return a.ctypes.data if a is not None else None


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {np.dtype(dtype)}, got {a.dtype}")
    return a


class Oracle:
    """numpy front end bound to one build of oracle.c."""

    def __init__(self, path):
        lib = ctypes.CDLL(path)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        self.lib = lib
        self.path = path

    def scan_i32(self, x, exclusive=False):
        """Inclusive (Section 2) or exclusive (Appendix B) int32 scan, mod 2^32."""
        x = _c(x, np.int32)
        y = np.empty(x.size, np.uint32)
        fn = self.lib.oracle_scan_exclusive_i32 if exclusive else self.lib.oracle_scan_inclusive_i32
        fn(_ptr(x), _ptr(y), x.size)
        return y.view(np.int32)

    def scan_f32(self, x, exclusive=False):
        """fp32 input scanned in float64.  Returns (prefix, prefix of |x|)."""
        x = _c(x, np.float32)
        y = np.empty(x.size, np.float64)
        a = np.empty(x.size, np.float64)
        fn = self.lib.oracle_scan_exclusive_f32 if exclusive else self.lib.oracle_scan_inclusive_f32
        fn(_ptr(x), _ptr(y), _ptr(a), x.size)
        return y, a

    def half_to_double(self, bits):
        """Decode one binary16 bit pattern exactly."""
        return self.lib.oracle_half_to_double(int(bits))

    def scan_f16(self, x, exclusive=False):
        """fp16 input (np.float16) scanned in float64.  Returns (prefix, |x| prefix)."""
        x = _c(x, np.float16).view(np.uint16)
        y = np.empty(x.size, np.float64)
        a = np.empty(x.size, np.float64)
        fn = self.lib.oracle_scan_exclusive_f16 if exclusive else self.lib.oracle_scan_inclusive_f16
        fn(_ptr(x), _ptr(y), _ptr(a), x.size)
        return y, a

    def scan_u8(self, x, exclusive=True):
        """8-bit values summed into int32 (mod 2^32).  Exclusive returns (y, total)."""
        x = _c(x, np.uint8)
        y = np.empty(x.size, np.uint32)
        if exclusive:
            total = ctypes.c_uint32(0)
            self.lib.oracle_scan_exclusive_u8(_ptr(x), _ptr(y), x.size, ctypes.addressof(total))
            return y.view(np.int32), int(np.uint32(total.value).view(np.int32))
        self.lib.oracle_scan_inclusive_u8(_ptr(x), _ptr(y), x.size)
        return y.view(np.int32)

    def scan_rows_i32(self, x, exclusive=False):
        """Independent int32 scan of every row of a 2-D array."""
        x = _c(x, np.int32)
        rows, length = x.shape
        y = np.empty((rows, length), np.uint32)
        self.lib.oracle_scan_rows_i32(_ptr(x), _ptr(y), rows, length, int(exclusive))
        return y.view(np.int32)

    def scan_rows_f32(self, x, exclusive=False):
        """Independent fp32 scan (float64 accumulation) of every row.  (y, |x| prefix)."""
        x = _c(x, np.float32)
        rows, length = x.shape
        y = np.empty((rows, length), np.float64)
        a = np.empty((rows, length), np.float64)
        self.lib.oracle_scan_rows_f32(_ptr(x), _ptr(y), _ptr(a), rows, length, int(exclusive))
        return y, a

    def compact_f32(self, x, mask):
        """Section 5 "Compress".  Returns (kept values, their source indices)."""
        x = _c(x, np.float32)
        mask = _c(mask, np.uint8)
        assert x.size == mask.size
        out = np.empty(x.size, np.float32)
        idx = np.empty(x.size, np.int32)
        c = self.lib.oracle_compact_f32(_ptr(x), _ptr(mask), _ptr(out), _ptr(idx), x.size)
        return out[:c].copy(), idx[:c].copy()

    def split_u32(self, keys, flags, idx_in=None):
        """Section 5 "Split".  Returns (keys_out, idx_out, n_true)."""
        keys = _c(keys, np.uint32)
        flags = _c(flags, np.uint8)
        assert keys.size == flags.size
        if idx_in is not None:
            idx_in = _c(idx_in, np.int32)
            assert idx_in.size == keys.size
        ko = np.empty(keys.size, np.uint32)
        io = np.empty(keys.size, np.int32)
        nt = self.lib.oracle_split_u32(_ptr(keys), _ptr(idx_in), _ptr(flags), _ptr(ko),
                                       _ptr(io), keys.size)
        return ko, io, int(nt)

    def sort_u32(self, keys):
        """Stable ascending sort of uint32 keys.  Returns (keys_out, perm)."""
        keys = _c(keys, np.uint32)
        ko = np.empty(keys.size, np.uint32)
        perm = np.empty(keys.size, np.int32)
        if self.lib.oracle_sort_u32(_ptr(keys), _ptr(ko), _ptr(perm), keys.size) != 0:
            raise MemoryError("oracle_sort_u32: allocation failed")
        return ko, perm

    def _sort_typed(self, name, keys, dtype, bits_dtype, descending):
        keys = _c(keys, dtype).view(bits_dtype)
        ko = np.empty(keys.size, bits_dtype)
        perm = np.empty(keys.size, np.int32)
        if getattr(self.lib, name)(_ptr(keys), _ptr(ko), _ptr(perm), keys.size,
                                   int(bool(descending))) != 0:
            raise MemoryError(f"{name}: allocation failed")
        return ko.view(dtype), perm

    def sort_i32(self, keys, descending=False):
        """Stable sort of int32 keys, ascending or descending.  Returns (keys_out, perm)."""
        return self._sort_typed("oracle_sort_i32", keys, np.int32, np.int32, descending)

    def sort_f32(self, keys, descending=False):
        """Stable sort of float32 keys in IEEE 754 totalOrder (bit copies)."""
        return self._sort_typed("oracle_sort_f32", keys, np.float32, np.uint32, descending)

    def sort_f16(self, keys, descending=False):
        """Stable sort of float16 keys in IEEE 754 totalOrder (bit copies)."""
        return self._sort_typed("oracle_sort_f16", keys, np.float16, np.uint16, descending)

    def sort_rows_f32(self, keys, descending=False):
        """Every row sorted on its own (stable, totalOrder); returns (keys_out, in-row idx)."""
        keys = _c(keys, np.float32)
        rows, length = keys.shape
        b = keys.view(np.uint32)
        ko = np.empty_like(b)
        idx = np.empty(keys.shape, np.int32)
        if self.lib.oracle_sort_rows_f32(_ptr(b), _ptr(ko), _ptr(idx), rows, length,
                                         int(bool(descending))) != 0:
            raise MemoryError("oracle_sort_rows_f32: allocation failed")
        return ko.view(np.float32), idx

    def weighted_sample_f32(self, w, theta):
        """Appendix "Weighted Sampling": per row, first i with S_i > theta * W."""
        w = _c(w, np.float32)
        rows, length = w.shape
        theta = _c(theta, np.float32)
        out = np.empty(rows, np.int32)
        self.lib.oracle_weighted_sample_f32(_ptr(w), _ptr(theta), _ptr(out), rows, length)
        return out

    def topp_sample_f32(self, probs, theta, p):
        """Section 5 "Top-p" sampler on unsorted rows: returns (token, cutoff) per row."""
        probs = _c(probs, np.float32)
        rows, length = probs.shape
        theta = _c(theta, np.float32)
        tok = np.empty(rows, np.int32)
        cut = np.empty(rows, np.int32)
        if self.lib.oracle_topp_sample_f32(_ptr(probs), _ptr(theta), float(p), _ptr(tok),
                                           _ptr(cut), rows, length) != 0:
            raise MemoryError("oracle_topp_sample_f32: allocation failed")
        return tok, cut

    def topk_rows_f32(self, x, k, largest=True):
        """Section 5 "Top-k": per row the k largest (or smallest) values in
        totalOrder, in order, ties by index.  Returns (values rows x k, in-row idx)."""
        x = _c(x, np.float32)
        rows, length = x.shape
        if not 0 <= k <= length:
            raise ValueError("k must be in [0, len]")
        vals = np.empty((rows, k), np.uint32)
        idx = np.empty((rows, k), np.int32)
        if self.lib.oracle_topk_rows_f32(_ptr(x.view(np.uint32)), _ptr(vals), _ptr(idx), rows,
                                         length, k, int(bool(largest))) != 0:
            raise MemoryError("oracle_topk_rows_f32: allocation failed")
        return vals.view(np.float32), idx

    def topp_cutoff_f32(self, probs, p):
        """Section 5 "Top-p": per row, first index whose float64 running sum >= p."""
        probs = _c(probs, np.float32)
        rows, length = probs.shape
        cut = np.empty(rows, np.int32)
        self.lib.oracle_topp_cutoff_f32(_ptr(probs), _ptr(cut), rows, length, float(p))
        return cut


_DEFAULT = None


def default() -> Oracle:
    """The oracle built from oracle/oracle.c (compiled on first use if absent)."""
    global _DEFAULT
    if _DEFAULT is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _DEFAULT = Oracle(_build.LIB)
    return _DEFAULT


def __getattr__(name):
    # module-level shortcuts: oracle.scan_i32(...) == oracle.default().scan_i32(...)
    if not name.startswith("_") and hasattr(Oracle, name):
        return getattr(default(), name)
    raise AttributeError(name)
