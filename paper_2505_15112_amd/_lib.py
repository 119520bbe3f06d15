"""ctypes loader for libscan.so: signatures mirror include/libscan.h exactly.

The library is loaded after ``import torch`` so that it binds to the HIP
runtime torch has already loaded (same soname) instead of a second copy; the
stream handles torch hands out are then valid inside the library.
"""
import contextlib
import ctypes
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libscan.so")
# the same sources with pseudo-random pauses before every inter-workgroup
# protocol step (adversarial-scheduling tests only)
LIB_ADV_PATH = os.path.join(PKG, "libscan_adv.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "libscan.h")

_p = ctypes.c_void_p
_i64 = ctypes.c_int64
_int = ctypes.c_int
_sz = ctypes.c_size_t

# name -> (restype, argtypes)
SIGNATURES = {
    "libscan_version": (_int, []),
    "libscan_status_string": (ctypes.c_char_p, [_int]),
    "libscan_workspace_bytes": (_int, [_int, _i64, _i64, _i64, _int, ctypes.POINTER(_sz)]),
    "libscan_workspace_init": (_int, [_p, _sz, _p]),
    "libscan_workspace_error": (_int, [_p, _sz, _p, _int, _p]),
    "scan_inclusive_i32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_exclusive_i32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_inclusive_f32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_exclusive_f32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_inclusive_f16f32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_exclusive_f16f32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_inclusive_f16f32_mfma": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_inclusive_f16f32_wave": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_exclusive_u8i32": (_int, [_p, _p, _i64, _p, _p, _sz, _p]),
    "scan_exclusive_u8i32_mfma": (_int, [_p, _p, _i64, _p, _p, _sz, _p]),
    "scan_exclusive_u8i32_wave": (_int, [_p, _p, _i64, _p, _p, _sz, _p]),
    "scan_inclusive_i32_carry": (_int, [_p, _p, _i64, _p, _p, _p, _sz, _p]),
    "scan_exclusive_i32_carry": (_int, [_p, _p, _i64, _p, _p, _p, _sz, _p]),
    "scan_inclusive_f32_carry": (_int, [_p, _p, _i64, _p, _p, _p, _sz, _p]),
    "scan_exclusive_f32_carry": (_int, [_p, _p, _i64, _p, _p, _p, _sz, _p]),
    "scan_inclusive_rss_i32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_inclusive_rss_f32": (_int, [_p, _p, _i64, _p, _sz, _p]),
    "scan_rows_i32": (_int, [_p, _p, _i64, _i64, _int, _p, _sz, _p]),
    "scan_rows_f32": (_int, [_p, _p, _i64, _i64, _int, _p, _sz, _p]),
    "topp_cutoff_f32": (_int, [_p, _p, _i64, _i64, ctypes.c_float, _p, _sz, _p]),
    "compact_by_mask_f32": (_int, [_p, _p, _p, _p, _p, _i64, _p, _sz, _p]),
    "split_by_flags_u32": (_int, [_p, _p, _p, _p, _p, _p, _i64, _p, _sz, _p]),
    "radix_sort_u32": (_int, [_p, _p, _p, _p, _p, _i64, _int, _p, _sz, _p]),
    "radix_sort_i32": (_int, [_p, _p, _p, _p, _p, _i64, _int, _p, _sz, _p]),
    "radix_sort_f32": (_int, [_p, _p, _p, _p, _p, _i64, _int, _p, _sz, _p]),
    "radix_sort_f16": (_int, [_p, _p, _p, _p, _p, _i64, _int, _p, _sz, _p]),
    "radix_sort_rows_f32": (_int, [_p, _p, _p, _p, _p, _i64, _i64, _int, _p, _sz, _p]),
    "weighted_sample_f32": (_int, [_p, _p, _p, _i64, _i64, _p, _sz, _p]),
    "topp_sample_f32": (_int, [_p, _p, ctypes.c_float, _p, _p, _i64, _i64, _p, _sz, _p, _sz,
                               _p]),
    "libscan_scratch_bytes": (_int, [_int, _i64, _i64, _i64, ctypes.POINTER(_sz)]),
    "topk_rows_f32": (_int, [_p, _p, _p, _i64, _i64, _i64, _int, _p, _sz, _p, _sz, _p]),
    "scan_inclusive_i32_noalloc": (_int, [_p, _p, _i64, _p]),
}

OK, EINVAL, ENOSPACE, EHIP, ERANGE = 0, -1, -2, -3, -4
OP_SCAN, OP_SCAN_RSS, OP_SCAN_ROWS, OP_COMPACT, OP_RADIX_SORT = 1, 2, 3, 4, 5
OP_SORT_ROWS, OP_WEIGHTED_SAMPLE, OP_TOPP_SAMPLE, OP_TOPK = 6, 7, 8, 9

_LIB = None


class LibscanError(RuntimeError):
    def __init__(self, name, status, lib):
        msg = lib.libscan_status_string(status).decode() if lib is not None else "?"
        super().__init__(f"{name} failed: {status} ({msg})")
        self.status = status


def header_functions(path: str = HEADER):
    """Names of the functions include/libscan.h declares."""
    text = open(path).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def load(path: str = LIB_PATH):
    """Load libscan.so once (after torch, see module docstring)."""
    global _LIB
    if _LIB is not None:
        return _LIB
    _LIB = _open(path)
    return _LIB


def _open(path: str):
    import torch  # noqa: F401  -- bind to torch's HIP runtime (see module docstring)
    if not os.path.exists(path):
        raise RuntimeError(
            f"{path} is not built; run `python -m paper_2505_15112_amd.build` "
            "(there is no fallback path)")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_ADV = None


def load_adversarial():
    """libscan_adv.so (see LIB_ADV_PATH), loaded once beside libscan.so."""
    global _ADV
    if _ADV is None:
        _ADV = _open(LIB_ADV_PATH)
    return _ADV


@contextlib.contextmanager
def using(lib):
    """Route every call made through this module to `lib` inside the block."""
    global _LIB
    load()
    saved = _LIB
    _LIB = lib
    try:
        yield lib
    finally:
        _LIB = saved


def call(name: str, *args):
    """Call an entry point; raise LibscanError on a non-zero status."""
    lib = load()
    st = getattr(lib, name)(*args)
    if st != OK:
        raise LibscanError(name, st, lib)
    return st


def scratch_bytes(op: int, rows: int, length: int, k: int = 0) -> int:
    lib = load()
    out = _sz(0)
    st = lib.libscan_scratch_bytes(op, rows, length, k, ctypes.byref(out))
    if st != OK:
        raise LibscanError("libscan_scratch_bytes", st, lib)
    return out.value


def workspace_bytes(op: int, n: int = 0, rows: int = 0, length: int = 0, bits: int = 0) -> int:
    lib = load()
    out = _sz(0)
    st = lib.libscan_workspace_bytes(op, n, rows, length, bits, ctypes.byref(out))
    if st != OK:
        raise LibscanError("libscan_workspace_bytes", st, lib)
    return out.value
