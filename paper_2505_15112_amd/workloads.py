"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random inputs (numpy ``default_rng``); it holds none of
the scan arithmetic and is the one piece of code that both the HIP path's
tests/benchmark and the CPU oracle's tests consume.  Every generator takes an
explicit seed and an integer stream tag, so two arrays of one workload come
from independent streams.

Recipes (the paper's workloads are synthetic; nothing here stands in for a
dataset):
  * 1-D int32 scan:       i.i.d. integers uniform on {0..100}
  * 1-D fp32 scan:        i.i.d. uniform on [-1, 1) in fp32
  * 1-D fp16 scan:        the fp32 draw rounded to fp16 (round to nearest even)
  * exact-float variant:  i.i.d. uniform on {-1, 0, 1}; every partial sum is an
                          integer far below 2^24, so any summation order is exact
  * mask / flags:         i.i.d. Bernoulli(1/2) bytes in {0, 1}  (Section 6,
                          "Compress": each mask entry true or false at random)
  * compaction values:    i.i.d. N(0, 1) fp32
  * top-p rows:           logits sigma * N(0, 1) per row, softmax in float64,
                          rounded to fp32, each row sorted descending
  * radix-sort keys:      i.i.d. uniform uint32 over [0, 2^32)
"""
import numpy as np


def _rng(seed: int, stream: int = 0) -> np.random.Generator:
    return np.random.default_rng([int(seed), int(stream)])


def scan_i32(n: int, seed: int = 0, stream: int = 0) -> np.ndarray:
    return _rng(seed, stream).integers(0, 101, size=n, dtype=np.int32)


def scan_i32_full_range(n: int, seed: int = 0, stream: int = 0) -> np.ndarray:
    """Any int32 bit pattern: exercises wrap-around modulo 2^32 heavily."""
    return _rng(seed, stream).integers(-2**31, 2**31, size=n, dtype=np.int32)


def scan_f32(n: int, seed: int = 0, stream: int = 0) -> np.ndarray:
    r = _rng(seed, stream).random(n, dtype=np.float32)
    return (r * np.float32(2.0) - np.float32(1.0)).astype(np.float32)


def scan_f16(n: int, seed: int = 0, stream: int = 0) -> np.ndarray:
    return scan_f32(n, seed, stream).astype(np.float16)


def exact_pm1(n: int, seed: int = 0, stream: int = 0, dtype=np.float32) -> np.ndarray:
    return _rng(seed, stream).integers(-1, 2, size=n, dtype=np.int8).astype(dtype)


def bytes_u8(n: int, seed: int = 0, stream: int = 0) -> np.ndarray:
    """Arbitrary byte values 0..255 (for the raw-byte-sum scan)."""
    return _rng(seed, stream).integers(0, 256, size=n, dtype=np.uint8)


def mask_u8(n: int, seed: int = 0, stream: int = 1, p_true: float = 0.5) -> np.ndarray:
    if p_true == 0.5:
        return _rng(seed, stream).integers(0, 2, size=n, dtype=np.uint8)
    return (_rng(seed, stream).random(n) < p_true).astype(np.uint8)


def values_f32(n: int, seed: int = 0, stream: int = 2) -> np.ndarray:
    return _rng(seed, stream).standard_normal(n, dtype=np.float32)


def keys_u32(n: int, seed: int = 0, stream: int = 3) -> np.ndarray:
    return _rng(seed, stream).integers(0, 2**32, size=n, dtype=np.uint32)


def topp_probs(rows: int, length: int, seed: int = 0, stream: int = 4,
               sigma: float = 2.0) -> np.ndarray:
    """Rows of a probability vector sorted descending (input preparation)."""
    rng = _rng(seed, stream)
    out = np.empty((rows, length), np.float32)
    for r in range(rows):
        z = sigma * rng.standard_normal(length)
        z -= z.max()
        e = np.exp(z)
        prob = (e / e.sum()).astype(np.float32)
        out[r] = -np.sort(-prob)
    return out


def sample_probs(rows: int, length: int, seed: int = 0, stream: int = 5,
                 sigma: float = 2.0) -> np.ndarray:
    """Rows of a probability vector in token order (unsorted): softmax of
    N(0, sigma^2) logits, as a sampler receives it."""
    rng = _rng(seed, stream)
    out = np.empty((rows, length), np.float32)
    for r in range(rows):
        z = sigma * rng.standard_normal(length)
        z -= z.max()
        e = np.exp(z)
        out[r] = (e / e.sum()).astype(np.float32)
    return out


def sample_theta(rows: int, seed: int = 0, stream: int = 6) -> np.ndarray:
    """One uniform draw in [0, 1) per row (float32)."""
    return _rng(seed, stream).random(rows, dtype=np.float32)


def sample_weights(rows: int, length: int, seed: int = 0, stream: int = 7,
                   zero_frac: float = 0.25) -> np.ndarray:
    """Non-negative unnormalised weights: exponential, a fraction exactly 0."""
    rng = _rng(seed, stream)
    w = rng.exponential(1.0, (rows, length)).astype(np.float32)
    w[rng.random((rows, length)) < zero_frac] = 0.0
    return w


# The workloads that tests and the benchmark use, by name.
METRIC_N = 1 << 28
CONFIGS = {
    "scan_i32_n2^16": dict(op="scan_inclusive_i32", n=1 << 16),
    "scan_f16f32_n2^24": dict(op="scan_inclusive_f16f32", n=1 << 24),
    "compact_n2^28": dict(op="compact_by_mask_f32", n=1 << 28),
    "topp_128x131072": dict(op="topp_cutoff_f32", rows=128, length=131072, p=0.9),
    "topp_sample_128x131072": dict(op="topp_sample_f32", rows=128, length=131072, p=0.9),
    "weighted_sample_128x131072": dict(op="weighted_sample_f32", rows=128, length=131072),
    "radix_n2^26": dict(op="radix_sort_u32", n=1 << 26),
    "metric_scan_n2^28": dict(op="scan_inclusive_i32/f32", n=METRIC_N),
}
