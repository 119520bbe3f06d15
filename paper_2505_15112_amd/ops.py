"""Tensor-level binding of libscan: argument marshalling only.

Each function checks dtype / device / contiguity, allocates missing outputs and
the workspace with torch (device memory plumbing), and calls the C entry point
of the same name on the current torch stream.  Every step of the computation
runs in libscan's HIP kernels; there is no fallback path.
"""
import ctypes

import torch

from . import _lib

_DT = {torch.int32: "i32", torch.float32: "f32", torch.float16: "f16", torch.uint8: "u8"}


def _check(t, dtype, name, dims=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: expected a GPU tensor, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if dims is not None and t.dim() not in dims:
        raise ValueError(f"{name}: expected {dims} dims, got {t.dim()}")


def _stream(dev):
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else None


def workspace(op: int, device, n: int = 0, rows: int = 0, length: int = 0, bits: int = 0):
    """A ready (zero-filled) device workspace big enough for op at these sizes.

    It can be reused by any later call of any op on the same stream."""
    nbytes = _lib.workspace_bytes(op, n, rows, length, bits)
    nbytes = max(16, (nbytes + 15) // 16 * 16)
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    with torch.cuda.device(ws.device):
        _lib.call("libscan_workspace_init", _ptr(ws), nbytes, _stream(ws.device))
    return ws


def _out(x, out, dtype, shape=None):
    shape = x.shape if shape is None else shape
    if out is None:
        return torch.empty(shape, dtype=dtype, device=x.device)
    _check(out, dtype, "out")
    if tuple(out.shape) != tuple(shape):
        raise ValueError(f"out: expected shape {tuple(shape)}, got {tuple(out.shape)}")
    return out


def _scan1d(cname, x, in_dtype, out_dtype, out, ws, extra=()):
    _check(x, in_dtype, "x")
    y = _out(x, out, out_dtype)
    n = x.numel()
    op = _lib.OP_SCAN_RSS if "_rss_" in cname else _lib.OP_SCAN
    if ws is None:
        ws = workspace(op, x.device, n)
    with torch.cuda.device(x.device):
        _lib.call(cname, _ptr(x), _ptr(y), n, *extra, _ptr(ws), ws.numel(), _stream(x.device))
    return y


def scan_inclusive_i32(x, out=None, ws=None):
    return _scan1d("scan_inclusive_i32", x, torch.int32, torch.int32, out, ws)


def scan_exclusive_i32(x, out=None, ws=None):
    return _scan1d("scan_exclusive_i32", x, torch.int32, torch.int32, out, ws)


def scan_inclusive_f32(x, out=None, ws=None):
    return _scan1d("scan_inclusive_f32", x, torch.float32, torch.float32, out, ws)


def scan_exclusive_f32(x, out=None, ws=None):
    return _scan1d("scan_exclusive_f32", x, torch.float32, torch.float32, out, ws)


def scan_inclusive_f16f32(x, out=None, ws=None):
    return _scan1d("scan_inclusive_f16f32", x, torch.float16, torch.float32, out, ws)


def scan_exclusive_f16f32(x, out=None, ws=None):
    return _scan1d("scan_exclusive_f16f32", x, torch.float16, torch.float32, out, ws)


def scan_exclusive_u8i32(x, out=None, total=None, ws=None):
    """Returns (y, total) -- total is a 1-element int32 device tensor."""
    if total is None:
        total = torch.empty(1, dtype=torch.int32, device=x.device)
    else:
        _check(total, torch.int32, "total")
    y = _scan1d("scan_exclusive_u8i32", x, torch.uint8, torch.int32, out, ws,
                extra=(ctypes.c_void_p(total.data_ptr()),))
    return y, total


def _carry(cname, dtype, x, carry_in, out, total_out, ws):
    if carry_in is not None:
        _check(carry_in, dtype, "carry_in")
    if total_out is None:
        total_out = torch.empty(1, dtype=dtype, device=x.device)
    else:
        _check(total_out, dtype, "total_out")
    cin = ctypes.c_void_p(carry_in.data_ptr()) if carry_in is not None else None
    y = _scan1d(cname, x, dtype, dtype, out, ws,
                extra=(cin, ctypes.c_void_p(total_out.data_ptr())))
    return y, total_out


def scan_inclusive_i32_carry(x, carry_in=None, out=None, total_out=None, ws=None):
    return _carry("scan_inclusive_i32_carry", torch.int32, x, carry_in, out, total_out, ws)


def scan_exclusive_i32_carry(x, carry_in=None, out=None, total_out=None, ws=None):
    return _carry("scan_exclusive_i32_carry", torch.int32, x, carry_in, out, total_out, ws)


def scan_inclusive_f32_carry(x, carry_in=None, out=None, total_out=None, ws=None):
    return _carry("scan_inclusive_f32_carry", torch.float32, x, carry_in, out, total_out, ws)


def scan_exclusive_f32_carry(x, carry_in=None, out=None, total_out=None, ws=None):
    return _carry("scan_exclusive_f32_carry", torch.float32, x, carry_in, out, total_out, ws)


def scan_inclusive_rss_i32(x, out=None, ws=None):
    return _scan1d("scan_inclusive_rss_i32", x, torch.int32, torch.int32, out, ws)


def scan_inclusive_rss_f32(x, out=None, ws=None):
    return _scan1d("scan_inclusive_rss_f32", x, torch.float32, torch.float32, out, ws)
