"""Tensor-level binding of libscan: argument marshalling only.

Each function checks dtype / device / contiguity, allocates missing outputs and
the workspace with torch (device memory plumbing), and calls the C entry point
of the same name on the current torch stream.  Every step of the computation
runs in libscan's HIP kernels; there is no fallback path.
"""
import ctypes
import os

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


def workspace_error(ws, reset=True):
    """The workspace's error word (0 or 1), read back to the host (this
    synchronises the stream); reset clears it.  1 means a call since the last
    reset gave up a bounded wait for another workgroup, so its outputs are
    unspecified (a workspace not zero-filled before first use, written by
    something else, or shared by concurrent calls)."""
    out = torch.zeros(1, dtype=torch.int32, device=ws.device)
    with torch.cuda.device(ws.device):
        _lib.call("libscan_workspace_error", _ptr(ws), ws.numel(),
                  ctypes.c_void_p(out.data_ptr()), int(bool(reset)), _stream(ws.device))
    return int(out.item())


# Checked mode: every call below then reads the workspace's error word after
# it (one stream synchronisation per call) and raises if it is set.
CHECKED = os.environ.get("LIBSCAN_CHECKED", "0") == "1"


def set_checked(on: bool):
    global CHECKED
    CHECKED = bool(on)


def _done(ws, name):
    if CHECKED and workspace_error(ws) != 0:
        raise _lib.LibscanError(name + " (workspace error word set)", _lib.EHIP, _lib.load())


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
        _done(ws, cname)
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


def scan_inclusive_f16f32_mfma(x, out=None, ws=None):
    """Inclusive fp16 -> fp32 scan with the row scans on the matrix cores."""
    return _scan1d("scan_inclusive_f16f32_mfma", x, torch.float16, torch.float32, out, ws)


def scan_inclusive_f16f32_wave(x, out=None, ws=None):
    """Inclusive fp16 -> fp32 scan on the wavefront tiles only."""
    return _scan1d("scan_inclusive_f16f32_wave", x, torch.float16, torch.float32, out, ws)


def _scan_u8(cname, x, out, total, ws):
    if total is None:
        total = torch.empty(1, dtype=torch.int32, device=x.device)
    else:
        _check(total, torch.int32, "total")
    y = _scan1d(cname, x, torch.uint8, torch.int32, out, ws,
                extra=(ctypes.c_void_p(total.data_ptr()),))
    return y, total


def scan_exclusive_u8i32(x, out=None, total=None, ws=None):
    """Returns (y, total) -- total is a 1-element int32 device tensor."""
    return _scan_u8("scan_exclusive_u8i32", x, out, total, ws)


def scan_exclusive_u8i32_mfma(x, out=None, total=None, ws=None):
    """The byte scan with the row scans on the matrix cores (x 16-byte aligned)."""
    return _scan_u8("scan_exclusive_u8i32_mfma", x, out, total, ws)


def scan_exclusive_u8i32_wave(x, out=None, total=None, ws=None):
    """The byte scan on the wavefront tiles only."""
    return _scan_u8("scan_exclusive_u8i32_wave", x, out, total, ws)


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


def _rows(cname, x, dtype, exclusive, out, ws):
    _check(x, dtype, "x", dims=(2,))
    rows, length = x.shape
    y = _out(x, out, dtype)
    if ws is None:
        ws = workspace(_lib.OP_SCAN_ROWS, x.device, rows=rows, length=length)
    with torch.cuda.device(x.device):
        _lib.call(cname, _ptr(x), _ptr(y), rows, length, int(bool(exclusive)), _ptr(ws),
                  ws.numel(), _stream(x.device))
        _done(ws, cname)
    return y


def scan_rows_i32(x, exclusive=False, out=None, ws=None):
    """Independent scan of every row of a 2-D int32 tensor."""
    return _rows("scan_rows_i32", x, torch.int32, exclusive, out, ws)


def scan_rows_f32(x, exclusive=False, out=None, ws=None):
    """Independent scan of every row of a 2-D fp32 tensor."""
    return _rows("scan_rows_f32", x, torch.float32, exclusive, out, ws)


def topp_cutoff_f32(probs, p, out=None, ws=None):
    """Per row of descending-sorted probabilities: first index whose running
    sum reaches p (int32 tensor of shape [rows])."""
    _check(probs, torch.float32, "probs", dims=(2,))
    rows, length = probs.shape
    cut = _out(probs, out, torch.int32, shape=(rows,))
    if ws is None:
        ws = workspace(_lib.OP_SCAN_ROWS, probs.device, rows=rows, length=length)
    with torch.cuda.device(probs.device):
        _lib.call("topp_cutoff_f32", _ptr(probs), _ptr(cut), rows, length, float(p), _ptr(ws),
                  ws.numel(), _stream(probs.device))
        _done(ws, "topp_cutoff_f32")
    return cut


def compact_by_mask_f32(x, mask, with_idx=False, out=None, idx_out=None, count=None, ws=None):
    """torch.masked_select order.  Returns (out, idx_out or None, count) with
    out/idx_out sized n (the first count entries are valid) and count a
    1-element int32 device tensor."""
    _check(x, torch.float32, "x")
    if mask.dtype == torch.bool:
        mask = mask.view(torch.uint8)
    _check(mask, torch.uint8, "mask")
    if mask.numel() != x.numel():
        raise ValueError("mask and x differ in size")
    n = x.numel()
    out = _out(x, out, torch.float32, shape=(n,))
    if with_idx and idx_out is None:
        idx_out = torch.empty(n, dtype=torch.int32, device=x.device)
    if count is None:
        count = torch.empty(1, dtype=torch.int32, device=x.device)
    if ws is None:
        ws = workspace(_lib.OP_COMPACT, x.device, n)
    with torch.cuda.device(x.device):
        _lib.call("compact_by_mask_f32", _ptr(x), _ptr(mask), _ptr(out), _ptr(idx_out),
                  ctypes.c_void_p(count.data_ptr()), n, _ptr(ws), ws.numel(), _stream(x.device))
        _done(ws, "compact_by_mask_f32")
    return out, idx_out, count


def split_by_flags_u32(keys, flags, idx_in=None, with_idx=True, keys_out=None, idx_out=None,
                       n_true=None, ws=None):
    """Stable split: flagged keys first.  keys are uint32 values held in an
    int32 tensor (torch has no uint32 arithmetic); returns
    (keys_out, idx_out or None, n_true)."""
    _check(keys, torch.int32, "keys")
    if flags.dtype == torch.bool:
        flags = flags.view(torch.uint8)
    _check(flags, torch.uint8, "flags")
    n = keys.numel()
    if flags.numel() != n:
        raise ValueError("flags and keys differ in size")
    if idx_in is not None:
        _check(idx_in, torch.int32, "idx_in")
    keys_out = _out(keys, keys_out, torch.int32, shape=(n,))
    if with_idx and idx_out is None:
        idx_out = torch.empty(n, dtype=torch.int32, device=keys.device)
    if n_true is None:
        n_true = torch.empty(1, dtype=torch.int32, device=keys.device)
    if ws is None:
        ws = workspace(_lib.OP_COMPACT, keys.device, n)
    with torch.cuda.device(keys.device):
        _lib.call("split_by_flags_u32", _ptr(keys), _ptr(idx_in), _ptr(flags), _ptr(keys_out),
                  _ptr(idx_out), ctypes.c_void_p(n_true.data_ptr()), n, _ptr(ws), ws.numel(),
                  _stream(keys.device))
        _done(ws, "split_by_flags_u32")
    return keys_out, idx_out, n_true


def radix_sort_u32(keys, bits_per_pass=8, with_perm=True, keys_out=None, perm_out=None,
                   keys_tmp=None, perm_tmp=None, ws=None):
    """Stable ascending sort of uint32 keys (held in an int32 tensor; compare
    them as unsigned), 1, 4 or 8 key bits per pass (8, the fewest passes, by
    default).  Returns (keys_out, perm_out or None)."""
    _check(keys, torch.int32, "keys")
    n = keys.numel()
    dev = keys.device
    keys_out = _out(keys, keys_out, torch.int32, shape=(n,))
    keys_tmp = torch.empty(n, dtype=torch.int32, device=dev) if keys_tmp is None else keys_tmp
    if with_perm:
        perm_out = torch.empty(n, dtype=torch.int32, device=dev) if perm_out is None else perm_out
        perm_tmp = torch.empty(n, dtype=torch.int32, device=dev) if perm_tmp is None else perm_tmp
    else:
        perm_out = perm_tmp = None
    if ws is None:
        ws = workspace(_lib.OP_RADIX_SORT, dev, n, bits=bits_per_pass)
    with torch.cuda.device(dev):
        _lib.call("radix_sort_u32", _ptr(keys), _ptr(keys_out), _ptr(perm_out), _ptr(keys_tmp),
                  _ptr(perm_tmp), n, int(bits_per_pass), _ptr(ws), ws.numel(), _stream(dev))
        _done(ws, "radix_sort_u32")
    return keys_out, perm_out


def _radix_sort_typed(cname, keys, dtype, descending, with_perm, keys_out, perm_out, keys_tmp,
                      perm_tmp, ws):
    _check(keys, dtype, "keys")
    n = keys.numel()
    dev = keys.device
    keys_out = _out(keys, keys_out, dtype, shape=(n,))
    keys_tmp = torch.empty(n, dtype=dtype, device=dev) if keys_tmp is None else keys_tmp
    if with_perm:
        perm_out = torch.empty(n, dtype=torch.int32, device=dev) if perm_out is None else perm_out
        perm_tmp = torch.empty(n, dtype=torch.int32, device=dev) if perm_tmp is None else perm_tmp
    else:
        perm_out = perm_tmp = None
    if ws is None:
        ws = workspace(_lib.OP_RADIX_SORT, dev, n, bits=8)
    with torch.cuda.device(dev):
        _lib.call(cname, _ptr(keys), _ptr(keys_out), _ptr(perm_out), _ptr(keys_tmp),
                  _ptr(perm_tmp), n, int(bool(descending)), _ptr(ws), ws.numel(), _stream(dev))
        _done(ws, cname)
    return keys_out, perm_out


def radix_sort_i32(keys, descending=False, with_perm=True, keys_out=None, perm_out=None,
                   keys_tmp=None, perm_tmp=None, ws=None):
    """Stable sort of int32 keys, ascending or descending.  Returns (keys_out, perm_out or None)."""
    return _radix_sort_typed("radix_sort_i32", keys, torch.int32, descending, with_perm, keys_out,
                             perm_out, keys_tmp, perm_tmp, ws)


def radix_sort_f32(keys, descending=False, with_perm=True, keys_out=None, perm_out=None,
                   keys_tmp=None, perm_tmp=None, ws=None):
    """Stable sort of float32 keys in IEEE 754 totalOrder (-NaN < -Inf < ... < -0 < +0 < ... <
    +Inf < +NaN), ascending or descending.  Returns (keys_out, perm_out or None)."""
    return _radix_sort_typed("radix_sort_f32", keys, torch.float32, descending, with_perm,
                             keys_out, perm_out, keys_tmp, perm_tmp, ws)


def radix_sort_f16(keys, descending=False, with_perm=True, keys_out=None, perm_out=None,
                   keys_tmp=None, perm_tmp=None, ws=None):
    """Stable sort of float16 keys in IEEE 754 totalOrder, ascending or descending."""
    return _radix_sort_typed("radix_sort_f16", keys, torch.float16, descending, with_perm,
                             keys_out, perm_out, keys_tmp, perm_tmp, ws)


def radix_sort_rows_f32(keys, descending=False, with_perm=True, keys_out=None, perm_out=None,
                        keys_tmp=None, perm_tmp=None, ws=None):
    """Stable sort of every row of a 2-D float32 tensor on its own (IEEE 754
    totalOrder).  perm_out holds indices within the row.  Returns (keys_out,
    perm_out or None)."""
    _check(keys, torch.float32, "keys", dims=(2,))
    rows, length = keys.shape
    dev = keys.device
    keys_out = _out(keys, keys_out, torch.float32)
    keys_tmp = torch.empty_like(keys) if keys_tmp is None else keys_tmp
    if with_perm:
        perm_out = _out(keys, perm_out, torch.int32)
        perm_tmp = torch.empty(keys.shape, dtype=torch.int32, device=dev) if perm_tmp is None \
            else perm_tmp
    else:
        perm_out = perm_tmp = None
    if ws is None:
        ws = workspace(_lib.OP_SORT_ROWS, dev, rows=rows, length=length)
    with torch.cuda.device(dev):
        _lib.call("radix_sort_rows_f32", _ptr(keys), _ptr(keys_out), _ptr(perm_out),
                  _ptr(keys_tmp), _ptr(perm_tmp), rows, length, int(bool(descending)), _ptr(ws),
                  ws.numel(), _stream(dev))
        _done(ws, "radix_sort_rows_f32")
    return keys_out, perm_out


def weighted_sample_f32(w, theta, out=None, ws=None):
    """Per row of non-negative weights: the index drawn by inverse transform
    with the uniform draw theta[row] (int32 tensor of shape [rows])."""
    _check(w, torch.float32, "w", dims=(2,))
    rows, length = w.shape
    _check(theta, torch.float32, "theta", dims=(1,))
    if theta.numel() != rows:
        raise ValueError(f"theta: expected {rows} draws, got {theta.numel()}")
    tok = _out(w, out, torch.int32, shape=(rows,))
    if ws is None:
        ws = workspace(_lib.OP_WEIGHTED_SAMPLE, w.device, rows=rows, length=length)
    with torch.cuda.device(w.device):
        _lib.call("weighted_sample_f32", _ptr(w), _ptr(theta), _ptr(tok), rows, length, _ptr(ws),
                  ws.numel(), _stream(w.device))
        _done(ws, "weighted_sample_f32")
    return tok


def scratch(op: int, device, rows: int, length: int, k: int = 0):
    """Scratch device memory for op at these sizes (no initialisation needed)."""
    nbytes = max(16, _lib.scratch_bytes(op, rows, length, k))
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def topp_sample_f32(probs, theta, p, with_cutoff=False, out=None, cutoff_out=None, ws=None,
                    scratch_buf=None):
    """Top-p sampling on unsorted rows: per row, the token drawn with the
    uniform draw theta[row] from the smallest descending-sorted prefix whose
    mass reaches p.  Returns the int32 tokens, and the cutoffs (index in the
    sorted row) when with_cutoff."""
    _check(probs, torch.float32, "probs", dims=(2,))
    rows, length = probs.shape
    _check(theta, torch.float32, "theta", dims=(1,))
    if theta.numel() != rows:
        raise ValueError(f"theta: expected {rows} draws, got {theta.numel()}")
    tok = _out(probs, out, torch.int32, shape=(rows,))
    cut = _out(probs, cutoff_out, torch.int32, shape=(rows,)) if with_cutoff else None
    if ws is None:
        ws = workspace(_lib.OP_TOPP_SAMPLE, probs.device, rows=rows, length=length)
    if scratch_buf is None:
        scratch_buf = scratch(_lib.OP_TOPP_SAMPLE, probs.device, rows, length)
    with torch.cuda.device(probs.device):
        _lib.call("topp_sample_f32", _ptr(probs), _ptr(theta), float(p), _ptr(tok), _ptr(cut),
                  rows, length, _ptr(scratch_buf), scratch_buf.numel(), _ptr(ws), ws.numel(),
                  _stream(probs.device))
        _done(ws, "topp_sample_f32")
    return (tok, cut) if with_cutoff else tok


def topk_rows_f32(x, k, largest=True, values_out=None, idx_out=None, ws=None, scratch_buf=None):
    """Per row of a 2-D float32 tensor, the k largest (or smallest) values in
    IEEE 754 totalOrder, in order, equal values by index.  Returns (values,
    int32 indices within the row), both rows x k."""
    _check(x, torch.float32, "x", dims=(2,))
    rows, length = x.shape
    k = int(k)
    vals = _out(x, values_out, torch.float32, shape=(rows, k))
    idx = _out(x, idx_out, torch.int32, shape=(rows, k))
    if ws is None:
        ws = workspace(_lib.OP_TOPK, x.device, k, rows=rows, length=length)
    if scratch_buf is None:
        scratch_buf = scratch(_lib.OP_TOPK, x.device, rows, length, k)
    with torch.cuda.device(x.device):
        _lib.call("topk_rows_f32", _ptr(x), _ptr(vals), _ptr(idx), rows, length, k,
                  int(bool(largest)), _ptr(scratch_buf), scratch_buf.numel(), _ptr(ws), ws.numel(),
                  _stream(x.device))
        _done(ws, "topk_rows_f32")
    return vals, idx
