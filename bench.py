#!/usr/bin/env python3
"""libscan benchmark on one MI355X.

One step = one 1-D inclusive prefix sum over n = 2^28 int32 elements (inputs
resident in HBM): the hot path's single kernel -- tile load, lane / wave /
workgroup scan, decoupled look-back, carry + store.  The printed value is the
achieved GB/s on the algorithmic bytes n*(4+4) (x read once, y written once),
beside a device-to-device memcpy of the same bytes timed in the same run, and
beside torch's elementwise streaming kernel over the same bytes (a higher bar:
it moves bytes faster than the runtime's memcpy).

The same run measures every other operation of the library on its workload
("ops"): the fp32 metric scan, the reduce-then-scan check variant, the
fp16->fp32 scan (n = 2^24), the latency-bound int32 scan (n = 2^16), mask
compaction (n = 2^28), batched rows and the top-p cutoff (128 x 131072),
the samplers on unsorted rows (top-p sampling, its descending row sort, and
weighted sampling, 128 x 131072), top-k of those rows (k = 64 and 4096),
stable split and the 1-, 4- and 8-bit radix sorts (n = 2^26).  Workloads
that fit in the 256 MB Infinity Cache are timed cold: rounds of (512 MiB
overwrite, call) enqueued back to back, minus the overwrites alone.
A sweep of the int32 scan over n = 2^20 .. 2^28 (and 2^k + 17) gives bandwidth
against length beside a memcpy of the same bytes; a sweep of batched fp32 row
scans of 2^16 elements over 16 .. 4096 rows the shape of the paper's
batched-scan experiment; the metric array scanned as 2^24-2^26-element
chunks through the carry entry points the analogue of its "L2 cache
splitting"; the fp16 radix sort with indices its radix-sort workload.
Every back-to-back row reports the batch's time per call and, from a second
batch with an event between calls, the median and minimum call; cold rows the
median and minimum of three rounds.  Every row but the metric (which takes the
--warmup calls it is given) warms up for at least 30 ms of GPU time first:
after the host-side pause of generating a row's inputs the GPU clock needs
about 10 ms of work to come back up.  After every row the workspace's error
word is read: a row whose bounded waits gave up fails the run.
The CPU-baseline leg times the serial oracle on each workload (or a stated
sample) and checks the GPU outputs against it (the samplers within the
acceptance band of their float readings).

--only ROW,... limits the measured rows (besides the metric) to those named.
Output: ONE JSON line on stdout.  --gpus N > 1 is refused: one GPU only.
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "scan GB/s (read+write) and % of same-run memcpy BW, 1-D n=2^28 int32/fp32"
PEAK_HBM_GBPS = 8000.0  # MI355X published HBM3E bandwidth
PMC_FILE = os.path.join(ROOT, "profiles", "scan_lookback_i32_n2^28_pmc.json")


METRIC_KERNEL_SOURCES = ("device.hpp", "tile.hpp", "scan1d.hip")


def kernel_source_hash() -> str:
    """sha256 over the sources of the metric kernel; ties counter measurements
    to the kernel version they were taken on."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2505_15112_amd", "csrc")
    for name in METRIC_KERNEL_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


TOPP_PMC_FILE = os.path.join(ROOT, "profiles", "topp_cutoff_128x131072_pmc.json")


def source_hash(names) -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2505_15112_amd", "csrc")
    for name in names:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


TOPP_KERNEL_SOURCES = ("device.hpp", "tile.hpp", "rowtile.hpp", "rows.hip")


def measured_topp_read():
    """HBM bytes the two top-p cutoff kernels read per call (rocprofv3
    FETCH_SIZE, scaled as for the metric), or None when absent or taken on
    other sources."""
    try:
        with open(TOPP_PMC_FILE) as f:
            pmc = json.load(f)
    except (OSError, ValueError):
        return None
    if pmc.get("kernel_source_sha256") != source_hash(TOPP_KERNEL_SOURCES):
        return None
    return pmc.get("hbm_read_bytes_per_call")


def measured_traffic():
    """HBM bytes per launch from the committed rocprofv3 PMC summary, or None
    when it is absent or was taken on different kernel sources."""
    try:
        with open(PMC_FILE) as f:
            pmc = json.load(f)
    except (OSError, ValueError):
        return None
    if pmc.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return pmc.get("hbm_bytes_per_launch")


class Stat(float):
    """A time in ms (the row's value) that also carries the median and the
    minimum of the individual measurements it came from."""

    def __new__(cls, value, median, minimum):
        s = float.__new__(cls, value)
        s.median, s.min = median, minimum
        return s


class Timer:
    def __init__(self, torch, stream, dev):
        self.torch = torch
        self.stream = stream
        self.flush_buf = torch.empty(512 << 20, dtype=torch.uint8, device=dev)

    def settle(self, body, calls, min_ms):
        """`calls` untimed calls of body, then more until about `min_ms` of GPU
        time has gone to warming up: after a host-side pause (input
        generation between rows) the GPU clock takes about 10 ms of work to
        ramp up again, and a few warm-up calls of a short op do not cover it
        (a 2^26-key 8-bit sort measured 1.20-1.29 ms for its first calls after
        an idle second, 1.15 ms once warm)."""
        torch = self.torch
        for _ in range(calls):
            body()
        if min_ms <= 0:
            return
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(self.stream)
        body()
        b.record(self.stream)
        torch.cuda.synchronize()
        one = max(a.elapsed_time(b), 1e-3)
        for _ in range(min(int(min_ms / one), 2000)):
            body()

    def back_to_back(self, fn, steps, warmup, min_warm_ms=0.0):
        """`steps` calls enqueued back to back between two events: the value
        is that batch's time per call.  A second batch of `steps` calls with
        an event between consecutive calls gives each call's own time, for the
        median and the minimum (kept apart so that those events cannot slow
        the batch the value comes from).  The per-op rows also warm up for
        at least min_warm_ms of GPU time (see settle); the metric takes the
        warm-up it is given."""
        torch = self.torch
        self.settle(fn, warmup, min_warm_ms)
        torch.cuda.synchronize()
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(self.stream)
        for _ in range(steps):
            fn()
        b.record(self.stream)
        torch.cuda.synchronize()
        mean = a.elapsed_time(b) / steps
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record(self.stream)
        for i in range(steps):
            fn()
            ev[i + 1].record(self.stream)
        torch.cuda.synchronize()
        per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
        return Stat(mean, per[len(per) // 2], per[0])

    def flushed(self, fn, steps, warmup, reps=3, min_warm_ms=30.0):
        """Cost of one call on data that is not in any cache: `steps` rounds of
        (overwrite 512 MiB, which evicts L2 and MALL; call) enqueued back to
        back, minus the same number of overwrites alone, per call; median of
        `reps`.  Timing each call alone between two events would add the
        event-to-kernel launch latency (about 6 us on MI355X) to every call."""
        torch = self.torch
        flush = self.flush_buf.zero_

        def both():
            flush()
            fn()

        self.settle(both, warmup, min_warm_ms)
        torch.cuda.synchronize()

        def timed(body):
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(self.stream)
            for _ in range(steps):
                body()
            b.record(self.stream)
            torch.cuda.synchronize()
            return a.elapsed_time(b)

        out = []
        for _ in range(reps):
            out.append((timed(both) - timed(flush)) / steps)
        out.sort()
        return Stat(out[len(out) // 2], out[len(out) // 2], out[0])


def device_info(torch, dev):
    """What the runtime reports about the GPU (no clocks: torch does not expose them)."""
    p = torch.cuda.get_device_properties(dev)
    return {"name": p.name, "arch": getattr(p, "gcnArchName", ""),
            "compute_units": p.multi_processor_count,
            "memory_gib": round(p.total_memory / 2**30, 1),
            "l2_bytes": getattr(p, "L2_cache_size", None),
            "hip": torch.version.hip}


def gpu_clocks():
    """Clock and power readings of the GPU from rocm-smi, or None."""
    import shutil
    import subprocess
    # Under a profiler its preloaded library initialises the GPU in every
    # child process, and rocm-smi's launcher hop (a script that re-execs its
    # interpreter) would then exec from such a process: skip the reading.
    if "rocprof" in os.environ.get("LD_PRELOAD", "") or any(
            k.startswith("ROCPROF") for k in os.environ):
        return None
    exe = shutil.which("rocm-smi") or "/opt/rocm/bin/rocm-smi"
    try:
        r = subprocess.run([exe, "--showclocks", "--showpower", "--json"], capture_output=True,
                           text=True, timeout=30)
        if r.returncode != 0:
            return None
        d = json.loads(r.stdout)
    except Exception:  # noqa: BLE001 -- a missing tool or odd output is just "not recorded"
        return None
    out = {}
    for card, vals in d.items():
        if isinstance(vals, dict):
            out[card] = {k: v for k, v in vals.items()
                         if any(t in k.lower() for t in ("clk", "clock", "power"))}
    return out or None


def host_cpu():
    """Model name and logical CPU count of the host the oracle runs on."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, os.cpu_count()


def entry(name, ms, nbytes, memcpy_ms, unit_note, extra=None, roof_bytes=None, roof_note=None):
    """One bench row.  nbytes: the algorithmic bytes (what the operation must
    read and write); the roofline is taken on roof_bytes when given (bytes the
    kernels were measured or counted to move, for kernels that read less than
    a full-size basis would credit)."""
    gbps = nbytes / (ms * 1e-3) / 1e9
    rb = nbytes if roof_bytes is None else roof_bytes
    rg = rb / (ms * 1e-3) / 1e9
    e = {"ms": round(ms, 5), "gbps": round(gbps, 2), "bytes": nbytes,
         "pct_of_memcpy": round(100.0 * memcpy_ms / ms, 2),
         "roofline": {"bound": "hbm", "achieved": round(rg, 2), "peak": PEAK_HBM_GBPS,
                      "unit": "GB/s", "frac": round(rg / PEAK_HBM_GBPS, 4)},
         "bytes_counted": unit_note}
    if roof_bytes is not None:
        e["roofline"]["bytes"] = roof_bytes
        e["roofline"]["bytes_basis"] = roof_note
    med, mn = getattr(ms, "median", None), getattr(ms, "min", None)
    if med is not None:
        e["ms_median"], e["ms_min"] = round(med, 5), round(mn, 5)
    if extra:
        e.update(extra)
    return e


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--n", type=int, default=1 << 28)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--metric-only", action="store_true", help="skip the per-op measurements")
    ap.add_argument("--only", default="", help="comma-separated rows to measure besides the "
                    "metric (batch, chunked, rss, f16, u8, c1, compact, topp, samplers, radix, "
                    "sweep); all by default")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: libscan is a single-GPU library; only --gpus 1 is supported "
              "(a sharded scan would exchange one carry per GPU).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2505_15112_amd import _lib, ops
    from paper_2505_15112_amd import workloads as W

    def log(*a):
        print("[bench]", *a, file=sys.stderr, flush=True)

    n = args.n
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    lib = _lib.load()
    sp = ctypes.c_void_p(stream.cuda_stream)
    T = Timer(torch, stream, dev)
    K, Wm = args.steps, args.warmup
    P = lambda t: ctypes.c_void_p(t.data_ptr()) if t is not None else None  # noqa: E731

    def check(st, name):
        if st != 0:
            raise RuntimeError(f"{name}: status {st}")

    err_buf = torch.zeros(1, dtype=torch.int32, device=dev)

    def ws_clean(w, name):
        """The workspace's error word after a row: 0, or the row is void."""
        check(lib.libscan_workspace_error(P(w), w.numel(), P(err_buf), 1, sp),
              "libscan_workspace_error")
        torch.cuda.synchronize()
        if int(err_buf.item()) != 0:
            raise RuntimeError(f"{name}: the workspace error word is set (a bounded wait gave up)")

    def memcpy_ms(nbytes, flushed=False):
        """D2D copy moving nbytes in total (nbytes/2 read + nbytes/2 written)."""
        m = max(1, nbytes // 2)
        src = torch.empty(m, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        f = lambda: dst.copy_(src)  # noqa: E731
        return (T.flushed(f, K, Wm) if flushed else T.back_to_back(f, K, Wm, 30.0))

    def streaming_ms(nbytes):
        """torch's elementwise kernel (int32 bitwise_not) moving nbytes in total: a
        plain streaming kernel, which moves bytes faster than the runtime's memcpy
        does, so a higher bar for the metric."""
        m = max(1, nbytes // 8)
        src = torch.zeros(m, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        return T.back_to_back(lambda: torch.bitwise_not(src, out=dst), K, Wm, 30.0)

    # ---------------------------------------------------------------- metric
    log("metric inputs")
    x_i32_host = W.scan_i32(n, seed=0)
    x_i32 = torch.from_numpy(x_i32_host).to(dev)
    y_i32 = torch.empty_like(x_i32)
    x_f32_host = W.scan_f32(n, seed=0)
    x_f32 = torch.from_numpy(x_f32_host).to(dev)
    y_f32 = torch.empty_like(x_f32)
    ws = ops.workspace(_lib.OP_SCAN, dev, n)
    wsp, wsb = P(ws), ws.numel()
    torch.cuda.synchronize()

    def scan_call(name, x, y, nn, w=None):
        fn = getattr(lib, name)
        wp, wb = (wsp, wsb) if w is None else (P(w), w.numel())
        a = (P(x), P(y), nn, wp, wb, sp)
        return lambda: check(fn(*a), name)

    nbytes = n * 8
    clocks_before = gpu_clocks()
    log("metric timing")
    ms_i32 = T.back_to_back(scan_call("scan_inclusive_i32", x_i32, y_i32, n), K, Wm)
    ms_f32 = T.back_to_back(scan_call("scan_inclusive_f32", x_f32, y_f32, n), K, Wm)
    ws_clean(ws, "metric")
    ms_cp = memcpy_ms(nbytes)
    ms_st = streaming_ms(nbytes)
    g = lambda ms, b=nbytes: b / (ms * 1e-3) / 1e9  # noqa: E731
    g_i32, g_f32, g_cp, g_st = g(ms_i32), g(ms_f32), g(ms_cp), g(ms_st)

    line = {
        "metric": METRIC,
        "value": round(g_i32, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(ms_i32, 4),
        "ms_per_step_median": round(ms_i32.median, 4),
        "ms_per_step_min": round(ms_i32.min, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i32",
        "data": "synthetic",
        "config": {
            "workload": "1-D inclusive prefix sum, n=2^28 int32, x_i iid uniform {0..100}",
            "n": n, "bytes_per_step": nbytes,
        },
        "device": device_info(torch, dev),
        "pct_of_memcpy": round(100.0 * g_i32 / g_cp, 2),
        "pct_of_peak_hbm": round(100.0 * g_i32 / PEAK_HBM_GBPS, 2),
        "memcpy_gbps": round(g_cp, 2),
        "pct_of_streaming_kernel": round(100.0 * g_i32 / g_st, 2),
        "streaming_kernel_gbps": round(g_st, 2),
        "fp32": {
            "value": round(g_f32, 2), "unit": "GB/s", "ms": round(ms_f32, 4),
            "ms_median": round(ms_f32.median, 4), "ms_min": round(ms_f32.min, 4),
            "workload": "1-D inclusive prefix sum, n=2^28 fp32, x_i iid uniform [-1,1)",
            "pct_of_memcpy": round(100.0 * g_f32 / g_cp, 2),
        },
        "roofline": {
            "kernel": "k_scan_lookback_lds<u32,19,9,16> (int32 inclusive, 114688-element tiles: "
                      "16 waves x (19 register + 9 LDS chunks of 1 KB), 16-byte vector path)",
            "bound": "hbm",
            "achieved": round(g_i32, 2),
            "peak": PEAK_HBM_GBPS,
            "unit": "GB/s",
            "frac": round(g_i32 / PEAK_HBM_GBPS, 4),
            "traffic": measured_traffic(),
            "algorithmic_bytes_per_launch": nbytes,
        },
    }

    # ---------------------------------------------------------------- other rows
    outputs = {}
    only = {w for w in args.only.split(",") if w}
    want = lambda k: not only or k in only  # noqa: E731
    if not args.metric_only:
        opsd = {}
        if want("batch"):
            # batched scans (appendix "Multiple (Batched) Scans"): rows of 2^16
            # elements over a growing batch, the shape of the paper's batched-scan
            # experiment (on the metric's fp32 input; cold below 512 MiB in all)
            log("batch sweep")
            wsb2 = ops.workspace(_lib.OP_SCAN_ROWS, dev, rows=n >> 16, length=1 << 16)
            batch = []
            for rows_b in (16, 64, 256, 1024, 4096):
                if rows_b << 16 > n:
                    continue
                xb2 = x_f32[: rows_b << 16]
                yb2 = y_f32[: rows_b << 16]
                a = (P(xb2), P(yb2), rows_b, 1 << 16, 0, P(wsb2), wsb2.numel(), sp)
                f = lambda a=a: check(lib.scan_rows_f32(*a), "rows")  # noqa: E731
                bb = (rows_b << 16) * 8
                cold = bb < (512 << 20)
                ms = T.flushed(f, K, Wm) if cold else T.back_to_back(f, K, Wm, 30.0)
                batch.append({"rows": rows_b, "len": 1 << 16, "us": round(ms * 1e3, 2),
                              "us_min": round(ms.min * 1e3, 2),
                              "gbps": round(bb / (ms * 1e-3) / 1e9, 1),
                              "pct_of_memcpy": round(100.0 * memcpy_ms(bb, cold) / ms, 1),
                              "cold": cold})
            ws_clean(wsb2, "batch sweep")
            line["batch_sweep_rows_f32_len2^16"] = batch
            del wsb2

        if want("chunked"):
            # chunked scans through the carry entry points (the analogue of the
            # paper's "L2 cache splitting", Section 6.1.1): the metric array as
            # consecutive chunks, each call adding the previous chunks' total
            log("chunked")
            cbuf = torch.zeros(1, dtype=torch.int32, device=dev)
            yc = torch.empty_like(x_i32)
            chunked = []
            for m in (1 << 24, 1 << 25, 1 << 26):
                def run_chunks(m=m):
                    for c0 in range(0, n, m):
                        st = lib.scan_inclusive_i32_carry(P(x_i32[c0:]), P(yc[c0:]), min(m, n - c0),
                                                          P(cbuf) if c0 else None, P(cbuf), wsp, wsb,
                                                          sp)
                        check(st, "scan_inclusive_i32_carry")
                ms = T.back_to_back(run_chunks, K, Wm, 30.0)
                chunked.append({"chunk": m, "chunks": n // m, "ms": round(ms, 4),
                                "ms_min": round(ms.min, 4), "gbps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                                "vs_one_call": round(ms_i32 / ms, 3),
                                "equal_to_one_call": bool(torch.equal(yc, y_i32))})
            ws_clean(ws, "chunked")
            line["chunked_carry_scan_i32_n2^28"] = chunked
            del yc, cbuf

        if want("rss"):
            # reduce-then-scan check variant (3 kernels, x read twice)
            wsr = ops.workspace(_lib.OP_SCAN_RSS, dev, n)
            y_rss = torch.empty_like(x_i32)
            ms = T.back_to_back(scan_call("scan_inclusive_rss_i32", x_i32, y_rss, n, wsr), K, Wm,
                                30.0)
            opsd["scan_rss_i32_n2^28"] = entry("rss", ms, nbytes, ms_cp, "n*(4+4); x is read twice",
                                              {"traffic_ratio_vs_lookback": 1.5})
            outputs["rss_equal"] = bool(torch.equal(y_rss, y_i32))
            ws_clean(wsr, "rss")
            del y_rss, wsr

        if want("f16"):
            # config: fp16 -> fp32, n = 2^24 (fits in MALL: flushed timing)
            n2 = 1 << 24
            x16_host = W.scan_f16(n2, seed=0)
            x16 = torch.from_numpy(x16_host).to(dev)
            y16 = torch.empty(n2, dtype=torch.float32, device=dev)
            b2 = n2 * 6
            ms = T.flushed(scan_call("scan_inclusive_f16f32", x16, y16, n2), K, Wm)
            opsd["scan_f16f32_n2^24"] = entry("f16", ms, b2, memcpy_ms(b2, True),
                                              "n*(2+4), cache-flushed; the default dispatch "
                                              "(wavefront tiles below n = 2^27)")
            outputs["f16"] = (x16_host, y16)
            # the same scan with its whole 32768-element tiles on the matrix
            # cores, cold at 2^24, and both forms back to back at 2^28 (where
            # the default takes the matrix cores)
            y16m = torch.empty_like(y16)
            ms = T.flushed(scan_call("scan_inclusive_f16f32_mfma", x16, y16m, n2), K, Wm)
            opsd["scan_f16f32_mfma_n2^24"] = entry("f16 mfma", ms, b2, memcpy_ms(b2, True),
                                                   "n*(2+4), cache-flushed; matrix-core tile scan")
            outputs["f16_mfma"] = (x16_host, y16m)
            x16b = torch.from_numpy(W.scan_f16(n, seed=3)).to(dev)
            y16b = torch.empty(n, dtype=torch.float32, device=dev)
            b28 = n * 6
            mc28 = memcpy_ms(b28)
            for nm in ("scan_inclusive_f16f32", "scan_inclusive_f16f32_wave"):
                ms = T.back_to_back(scan_call(nm, x16b, y16b, n), K, Wm, 30.0)
                key = "scan_f16f32" + ("_wave" if nm.endswith("wave") else "") + "_n2^28"
                opsd[key] = entry("f16 2^28", ms, b28, mc28, "n*(2+4)")
            del x16b, y16b

        if want("u8"):
            # the exclusive byte scan (mask counts), n = 2^28: the default
            # wavefront tiles against the matrix-core variant, 1 + 4 bytes per element
            xb = torch.from_numpy(W.mask_u8(n, seed=4)).to(dev)
            yb = torch.empty(n, dtype=torch.int32, device=dev)
            tb = torch.empty(1, dtype=torch.int32, device=dev)
            b5 = n * 5
            mc5 = memcpy_ms(b5)
            for nm in ("scan_exclusive_u8i32", "scan_exclusive_u8i32_mfma"):
                fn = getattr(lib, nm)
                a = (P(xb), P(yb), n, P(tb), wsp, wsb, sp)
                ms = T.back_to_back(lambda: check(fn(*a), nm), K, Wm, 30.0)
                key = "scan_u8i32" + ("_mfma" if nm.endswith("mfma") else "") + "_n2^28"
                opsd[key] = entry("u8", ms, b5, mc5, "n*(1+4)")
            ws_clean(ws, "scans")
            del xb, yb, tb

        if want("c1"):
            # config: int32, n = 2^16 (latency-bound)
            n1 = 1 << 16
            x1_host = W.scan_i32(n1, seed=0)
            x1 = torch.from_numpy(x1_host).to(dev)
            y1 = torch.empty_like(x1)
            ms_f = T.flushed(scan_call("scan_inclusive_i32", x1, y1, n1), K, Wm)
            ms_b = T.back_to_back(scan_call("scan_inclusive_i32", x1, y1, n1), K, Wm, 30.0)
            opsd["scan_i32_n2^16"] = entry("c1", ms_f, n1 * 8, memcpy_ms(n1 * 8, True),
                                           "n*(4+4), cache-flushed; latency-bound",
                                           {"us_flushed": round(ms_f * 1e3, 2),
                                            "us_back_to_back": round(ms_b * 1e3, 2)})
            outputs["c1"] = (x1_host, y1)

        if want("compact"):
            # config: compaction n = 2^28, Bernoulli(1/2) mask, N(0,1) values
            log("compaction")
            vals_host = W.values_f32(n, seed=0)
            mask_host = W.mask_u8(n, seed=0)
            vals = torch.from_numpy(vals_host).to(dev)
            mask = torch.from_numpy(mask_host).to(dev)
            out = torch.empty_like(vals)
            idx = torch.empty(n, dtype=torch.int32, device=dev)
            cnt = torch.empty(1, dtype=torch.int32, device=dev)
            wsc = ops.workspace(_lib.OP_COMPACT, dev, n)
            fnc = lib.compact_by_mask_f32
            for with_idx in (False, True):
                a = (P(vals), P(mask), P(out), P(idx) if with_idx else None, P(cnt), n, P(wsc),
                     wsc.numel(), sp)
                ms = T.back_to_back(lambda: check(fnc(*a), "compact"), K, Wm, 30.0)
                c = int(cnt.item())
                bb = n * 5 + c * 4 + (c * 4 if with_idx else 0)
                opsd["compact_n2^28" + ("_idx" if with_idx else "")] = entry(
                    "compact", ms, bb, memcpy_ms(bb), "n*(1+4) + count*4 (+count*4 indices)",
                    {"count": c})
            outputs["compact"] = (vals_host, mask_host, out, idx, cnt)
            ws_clean(wsc, "compact")
        del x_f32, y_f32

        rows, length = 128, 131072
        bt = rows * length * 4
        if want("topp"):
            # config: rows + top-p, 128 x 131072 sorted softmax rows (64 MiB: flushed)
            log("rows/top-p")
            probs_host = W.topp_probs(rows, length, seed=0)
            probs = torch.from_numpy(probs_host).to(dev)
            cut = torch.empty(rows, dtype=torch.int32, device=dev)
            wst = ops.workspace(_lib.OP_SCAN_ROWS, dev, rows=rows, length=length)
            a = (P(probs), P(cut), rows, length, ctypes.c_float(0.9), P(wst), wst.numel(), sp)
            ms = T.flushed(lambda: check(lib.topp_cutoff_f32(*a), "topp"), K, Wm)
            ws_clean(wst, "topp")
            # algorithmic: the prefix of each row up to its cutoff (what the
            # definition must read) and the cutoffs.  The kernels read the row
            # heads (a quarter of each row, at least 8 tiles of 4096) and re-read
            # one tile per row from L2; rocprofv3's FETCH_SIZE of the same call,
            # when taken on these sources, is the roofline's basis.
            kq = cut.cpu().numpy().astype(np.int64)
            alg = int(np.sum(kq + 1)) * 4 + rows * 4
            segs = -(-length // 4096)
            heads = min(segs, max(8, -(-segs // 4)))
            read = rows * heads * 4096 * 4 + rows * 4096 * 4
            fetch = measured_topp_read()
            opsd["topp_128x131072"] = entry(
                "topp", ms, alg, memcpy_ms(bt, True),
                "each row's prefix up to its cutoff + the cutoffs (rows*(cutoff+1)*4 + rows*4), "
                "cache-flushed; memcpy of the full rows",
                {"p": 0.9, "bytes_full_rows": bt, "bytes_read_by_kernels": read,
                 "bytes_fetch_counter": fetch, "heads_tiles": heads,
                 "cutoffs_in_head": bool(np.all(kq < heads * 4096))},
                roof_bytes=fetch if fetch else read,
                roof_note="rocprofv3 FETCH_SIZE per call" if fetch else
                "bytes the kernels read (heads + one re-read tile per row)")
            yr = torch.empty_like(probs)
            a2 = (P(probs), P(yr), rows, length, 0, P(wst), wst.numel(), sp)
            ms = T.flushed(lambda: check(lib.scan_rows_f32(*a2), "rows"), K, Wm)
            opsd["scan_rows_f32_128x131072"] = entry("rows", ms, 2 * bt, memcpy_ms(2 * bt, True),
                                                     "rows*len*(4+4), cache-flushed")
            ws_clean(wst, "rows")
            outputs["topp"] = (probs_host, cut, yr)

        if want("samplers"):
            # config: the samplers on 128 x 131072 unsorted softmax rows (one draw per row)
            log("samplers")
            sp_host = W.sample_probs(rows, length, seed=0)
            th_host = W.sample_theta(rows, seed=0)
            sprobs = torch.from_numpy(sp_host).to(dev)
            theta = torch.from_numpy(th_host).to(dev)
            tok = torch.empty(rows, dtype=torch.int32, device=dev)
            cut2 = torch.empty(rows, dtype=torch.int32, device=dev)
            ws_smp = ops.workspace(_lib.OP_TOPP_SAMPLE, dev, rows=rows, length=length)
            scr = ops.scratch(_lib.OP_TOPP_SAMPLE, dev, rows, length)
            a = (P(sprobs), P(theta), ctypes.c_float(0.9), P(tok), P(cut2), rows, length, P(scr),
                 scr.numel(), P(ws_smp), ws_smp.numel(), sp)
            ms = T.flushed(lambda: check(lib.topp_sample_f32(*a), "topp sample"), K, Wm)
            # the descending sort with indices (4 passes: 12 + 16 x 3 + 4 bytes per key) and one
            # read of the sorted row
            bb = rows * length * (64 + 4)
            opsd["topp_sample_128x131072"] = entry(
                "topp_sample", ms, bb, memcpy_ms(bb, True),
                "rows*len*(64 sort + 4 draw), cache-flushed",
                {"p": 0.9, "draws_per_s": round(rows / (ms * 1e-3), 1)})
            ko2 = torch.empty_like(sprobs)
            po2 = torch.empty(rows, length, dtype=torch.int32, device=dev)
            kt2 = torch.empty_like(sprobs)
            pt2 = torch.empty_like(po2)
            a = (P(sprobs), P(ko2), P(po2), P(kt2), P(pt2), rows, length, 1, P(ws_smp), ws_smp.numel(), sp)
            ms = T.flushed(lambda: check(lib.radix_sort_rows_f32(*a), "sort rows"), K, Wm)
            bb = rows * length * 64
            opsd["sort_rows_f32_desc_128x131072"] = entry(
                "sort_rows", ms, bb, memcpy_ms(bb, True), "rows*len*(12 + 16 x 3 + 4), cache-flushed",
                {"mkeys_per_s": round(rows * length / (ms * 1e-3) / 1e6, 1)})
            wtok = torch.empty(rows, dtype=torch.int32, device=dev)
            a = (P(sprobs), P(theta), P(wtok), rows, length, P(ws_smp), ws_smp.numel(), sp)
            ms = T.flushed(lambda: check(lib.weighted_sample_f32(*a), "weighted"), K, Wm)
            opsd["weighted_sample_128x131072"] = entry(
                "weighted_sample", ms, bt, memcpy_ms(bt, True),
                "weights read once (rows*len*4), cache-flushed",
                {"draws_per_s": round(rows / (ms * 1e-3), 1)})
            outputs["samplers"] = (sp_host, th_host, tok, cut2, wtok)
            ws_clean(ws_smp, "samplers")
            # top-k of the same rows.  Algorithmic: one read of each row and the k
            # values and indices written per row.  For k <= 256 the implementation
            # reads each row once (every tile keeps its keys at or above its own
            # k-th key's top 16 bits); for larger k it reads the rows twice (one
            # digit-count round, then the gather of the keys at or above the
            # k-th's top byte).  Either way the candidates are then selected and
            # ordered per row in LDS: reported beside it, without the
            # candidates' own bytes (8 B written and read back per candidate, a
            # few thousand per row).
            topk_out = {}
            for kq in (64, 4096):
                wsk = ops.workspace(_lib.OP_TOPK, dev, kq, rows=rows, length=length)
                sck = ops.scratch(_lib.OP_TOPK, dev, rows, length, kq)
                tv = torch.empty(rows, kq, dtype=torch.float32, device=dev)
                ti = torch.empty(rows, kq, dtype=torch.int32, device=dev)
                a = (P(sprobs), P(tv), P(ti), rows, length, kq, 1, P(sck), sck.numel(), P(wsk),
                     wsk.numel(), sp)
                ms = T.flushed(lambda: check(lib.topk_rows_f32(*a), "topk"), K, Wm)
                ws_clean(wsk, "topk")
                bb = rows * length * 4 + rows * kq * 8
                reads = 1 if kq <= 256 else 2
                impl = rows * length * 4 * reads + rows * kq * 8
                opsd[f"topk_k{kq}_128x131072"] = entry(
                    "topk", ms, bb, memcpy_ms(bb, True),
                    "rows*len*4 (one read of each row) + rows*k*8 (values and indices), "
                    "cache-flushed",
                    {"k": kq, "rows_per_s": round(rows / (ms * 1e-3), 1),
                     "bytes_moved_by_implementation": impl,
                     "implementation_bytes_counted": (
                         "rows*len*4 (one read: tile selection) + rows*k*8 (values and indices)"
                         if reads == 1 else
                         "rows*len*(4 counting + 4 gather) + rows*k*8 (values and indices)"),
                     "gbps_on_implementation_bytes": round(impl / (ms * 1e-3) / 1e9, 2)})
                topk_out[kq] = (tv, ti)
                del wsk, sck
            outputs["topk"] = topk_out
            del ko2, po2, kt2, pt2, scr

        if want("radix"):
            # config: radix sort, n = 2^26 uint32 keys (+ int32 permutation)
            log("radix")
            n5 = 1 << 26
            keys_host = W.keys_u32(n5, seed=0)
            keys = torch.from_numpy(keys_host.view(np.int32)).to(dev)
            ko = torch.empty_like(keys)
            po = torch.empty_like(keys)
            kt = torch.empty_like(keys)
            pt = torch.empty_like(keys)
            for bits, passes in ((8, 4), (4, 8), (1, 32)):
                wsx = ops.workspace(_lib.OP_RADIX_SORT, dev, n5, bits=bits)
                a = (P(keys), P(ko), P(po), P(kt), P(pt), n5, bits, P(wsx), wsx.numel(), sp)
                ms = T.back_to_back(lambda: check(lib.radix_sort_u32(*a), "radix"), max(3, K // 4),
                                    2, 30.0)
                # algorithmic bytes: pass 0 reads keys and writes keys + indices (12 B),
                # later passes read and write both (16 B); the 4- and 8-bit sorts also
                # need one histogram read (4 B).  Reads this implementation adds (the
                # 1-bit histogram, the per-pass count kernels) are not credited.
                bb = n5 * (12 + 16 * (passes - 1) + (4 if bits > 1 else 0))
                opsd[f"radix{bits}_n2^26"] = entry(
                    "radix", ms, bb, memcpy_ms(bb), "12 + 16 x (passes-1) bytes per key"
                    + (" + 4 (histogram)" if bits > 1 else ""),
                    {"mkeys_per_s": round(n5 / (ms * 1e-3) / 1e6, 1), "passes": passes})
                outputs[f"radix{bits}"] = (ko.clone(), po.clone())
                ws_clean(wsx, f"radix{bits}")
            # float32 keys, descending (the top-p sampler's order), 8-bit digits
            kf = torch.from_numpy(W.values_f32(n5, seed=2)).to(dev)
            kfo = torch.empty_like(kf)
            kft = torch.empty_like(kf)
            wsx = ops.workspace(_lib.OP_RADIX_SORT, dev, n5, bits=8)
            a = (P(kf), P(kfo), P(po), P(kft), P(pt), n5, 1, P(wsx), wsx.numel(), sp)
            ms = T.back_to_back(lambda: check(lib.radix_sort_f32(*a), "radix f32"), max(3, K // 4),
                                2, 30.0)
            bb = n5 * (12 + 16 * 3 + 4)
            opsd["radix8_f32_desc_n2^26"] = entry(
                "radix", ms, bb, memcpy_ms(bb), "12 + 16 x 3 + 4 bytes per key (4 passes)",
                {"mkeys_per_s": round(n5 / (ms * 1e-3) / 1e6, 1), "passes": 4})
            del kf, kfo, kft
            # float16 keys with indices, ascending: the paper's radix-sort workload
            # (Section 6 sorts fp16 keys and returns indices); 8-bit digits, so 2
            # passes: pass 0 reads keys and writes keys + indices (2 + 2 + 4 B),
            # pass 1 reads and writes both (2 * 6 B)
            kh16 = W.scan_f16(n5, seed=5)
            k16 = torch.from_numpy(kh16).to(dev)
            k16o = torch.empty_like(k16)
            k16t = torch.empty_like(k16)
            a = (P(k16), P(k16o), P(po), P(k16t), P(pt), n5, 0, P(wsx), wsx.numel(), sp)
            ms = T.back_to_back(lambda: check(lib.radix_sort_f16(*a), "radix f16"), max(3, K // 4),
                                2, 30.0)
            bb = n5 * (8 + 12)
            opsd["radix8_f16_n2^26"] = entry(
                "radix", ms, bb, memcpy_ms(bb), "8 + 12 bytes per key (2 passes of 16-bit keys and "
                "int32 indices)", {"mkeys_per_s": round(n5 / (ms * 1e-3) / 1e6, 1), "passes": 2})
            outputs["radix_f16"] = (kh16, k16o.clone(), po.clone())
            ws_clean(wsx, "radix f16")
            del k16, k16o, k16t

            # stable split on its own (flags Bernoulli(1/2)), n = 2^26
            flags = torch.from_numpy(W.mask_u8(n5, seed=1)).to(dev)
            nt = torch.empty(1, dtype=torch.int32, device=dev)
            wss = ops.workspace(_lib.OP_COMPACT, dev, n5)
            a = (P(keys), None, P(flags), P(ko), P(po), P(nt), n5, P(wss), wss.numel(), sp)
            ms = T.back_to_back(lambda: check(lib.split_by_flags_u32(*a), "split"), K, Wm, 30.0)
            bb = n5 * (1 + 1 + 4 + 4 + 4)  # count kernel reads flags; split reads flags+keys, writes
            opsd["split_n2^26"] = entry("split", ms, bb, memcpy_ms(bb), "n*(1 count + 1+4 read + "
                                        "4+4 written), no input indices")
            ws_clean(wss, "split")
            outputs["radix_keys"] = keys_host

        line["ops"] = opsd

        if want("sweep"):
            # bandwidth against length, int32 inclusive: powers of two and 2^k + 17
            # (ragged last tile); totals under 512 MiB are timed cold
            log("sweep")
            sweep = []
            for k in range(20, 29):
                for m in (1 << k, (1 << k) + 17):
                    if m > n:
                        continue
                    xs, ys = x_i32[:m], y_i32[:m]
                    cold = m * 8 < (512 << 20)
                    f = scan_call("scan_inclusive_i32", xs, ys, m)
                    ms = T.flushed(f, K, Wm) if cold else T.back_to_back(f, K, Wm, 30.0)
                    mc = memcpy_ms(m * 8, cold)
                    sweep.append({"n": m, "us": round(ms * 1e3, 2),
                                  "gbps": round(m * 8 / (ms * 1e-3) / 1e9, 1),
                                  "pct_of_memcpy": round(100.0 * mc / ms, 1), "cold": cold})
            line["sweep_i32"] = sweep
            ws_clean(ws, "sweep")
    line["gpu_clocks"] = {"before_metric": clocks_before, "after": gpu_clocks()}

    # ---------------------------------------------------------------- CPU leg
    if not args.no_cpu_baseline:
        log("cpu baseline")
        line["cpu_baseline"], line["cpu_baseline_ops"] = cpu_baseline_leg(
            x_i32_host, y_i32, outputs, np, torch)
    print(json.dumps(line), flush=True)
    return 0


def cpu_baseline_leg(x_host, y_dev, outputs, np, torch):
    """The serial CPU oracle timed on the machine's host (one thread), and every
    GPU output of this run checked against it."""
    import oracle

    def timed(fn, reps=3):
        ts, r = [], None
        for _ in range(reps):
            t0 = time.perf_counter()
            r = fn()
            ts.append(time.perf_counter() - t0)
        return sorted(ts)[len(ts) // 2], r

    t, ref = timed(lambda: oracle.scan_i32(x_host))
    metric = {
        "value": round(x_host.size * 8 / t / 1e9, 3), "unit": "GB/s", "cores": 1,
        "kind": "oracle",
        "sample": f"the full workload: 1-D inclusive int32 scan of n={x_host.size} "
                  f"(serial C oracle, median of 3 runs, {t:.3f} s each)",
        "matches_gpu": bool(np.array_equal(ref, y_dev.cpu().numpy())),
    }
    metric["host_cpu_model"], metric["host_logical_cpus"] = host_cpu()
    res = {}
    if "f16" in outputs:
        xh, y = outputs["f16"]
        t, (r, a) = timed(lambda: oracle.scan_f16(xh))
        ok = bool(np.all(np.abs(y.cpu().numpy() - r) <= 1e-5 * a + 1e-6))
        res["scan_f16f32_n2^24"] = {"gbps": round(xh.size * 6 / t / 1e9, 3), "s": round(t, 4),
                                    "matches_gpu": ok}
        xh, y = outputs["f16_mfma"]
        res["scan_f16f32_mfma_n2^24"] = {
            "matches_gpu": bool(np.all(np.abs(y.cpu().numpy() - r) <= 1e-5 * a + 1e-6))}
    if "c1" in outputs:
        xh, y = outputs["c1"]
        t, r = timed(lambda: oracle.scan_i32(xh))
        res["scan_i32_n2^16"] = {"us": round(t * 1e6, 1),
                                 "matches_gpu": bool(np.array_equal(r, y.cpu().numpy()))}
    if "rss_equal" in outputs:
        res["scan_rss_i32_n2^28"] = {"matches_lookback_bitwise": outputs["rss_equal"]}
    if "compact" in outputs:
        vh, mh, out, idx, cnt = outputs["compact"]
        t, (ro, ri) = timed(lambda: oracle.compact_f32(vh, mh), reps=1)
        c = int(cnt.item())
        ok = c == ro.size and np.array_equal(out[:c].cpu().numpy().view(np.uint32),
                                             ro.view(np.uint32)) and np.array_equal(
            idx[:c].cpu().numpy(), ri)
        res["compact_n2^28"] = {"gbps": round((vh.size * 5 + c * 8) / t / 1e9, 3),
                                "s": round(t, 3), "matches_gpu": bool(ok)}
    if "topp" in outputs:
        ph, cut, yr = outputs["topp"]
        t, rc = timed(lambda: oracle.topp_cutoff_f32(ph, 0.9))
        g = cut.cpu().numpy()
        csum = np.cumsum(ph.astype(np.float64), axis=1)
        tol = 1e-5 * csum + 1e-6
        pd = float(np.float32(0.9))
        band = [g[r] == rc[r] or (csum[r, g[r]] >= pd - tol[r, g[r]] and
                                  (g[r] == 0 or csum[r, g[r] - 1] < pd + tol[r, g[r] - 1]))
                for r in range(ph.shape[0])]
        res["topp_128x131072"] = {"gbps": round(ph.size * 4 / t / 1e9, 3), "s": round(t, 4),
                                  "matches_gpu_within_band": bool(all(band)),
                                  "exact_rows": int(np.sum(g == rc))}
        t, (ry, ra) = timed(lambda: oracle.scan_rows_f32(ph), reps=1)
        ok = bool(np.all(np.abs(yr.cpu().numpy() - ry) <= 1e-5 * ra + 1e-6))
        res["scan_rows_f32_128x131072"] = {"gbps": round(ph.size * 8 / t / 1e9, 3),
                                           "s": round(t, 4), "matches_gpu": ok}
    if "samplers" in outputs:
        # the samplers against the oracle: equal, or inside the acceptance band
        # of readings A15 (cutoff) and A22 (draw) -- the same test as the GPU
        # parity tests apply
        sys.path.insert(0, os.path.join(ROOT, "tests"))
        from gpu_util import draw_accept, draw_tol, topp_accept
        ph, th, tok, cut2, wtok = outputs["samplers"]
        t, (rt, rc) = timed(lambda: oracle.topp_sample_f32(ph, th, 0.9), reps=1)
        g, gc = tok.cpu().numpy(), cut2.cpu().numpy()
        sk, sp_ = oracle.sort_rows_f32(ph, descending=True)
        band = []
        for r in range(ph.shape[0]):
            if g[r] == rt[r] and gc[r] == rc[r]:
                band.append(True)
                continue
            scs = np.cumsum(sk[r].astype(np.float64))
            k = int(gc[r])
            jj = np.flatnonzero(sp_[r] == g[r])
            ok = topp_accept(k, int(rc[r]), scs, 0.9) and jj.size == 1 and draw_accept(
                int(jj[0]), scs, float(th[r]) * float(scs[k]), draw_tol(float(th[r]),
                                                                       float(scs[k])), k)
            band.append(bool(ok))
        res["topp_sample_128x131072"] = {
            "draws_per_s": round(ph.shape[0] / t, 1), "s": round(t, 3),
            "exact_rows": int(np.sum((g == rt) & (gc == rc))), "rows": int(ph.shape[0]),
            "matches_gpu_within_band": bool(all(band))}
        t, rw = timed(lambda: oracle.weighted_sample_f32(ph, th))
        gw = wtok.cpu().numpy()
        band = []
        for r in range(ph.shape[0]):
            cs = np.cumsum(ph[r].astype(np.float64))
            tot = float(cs[-1])
            band.append(bool(gw[r] == rw[r] or draw_accept(
                int(gw[r]), cs, float(th[r]) * tot, draw_tol(float(th[r]), tot), ph.shape[1] - 1)))
        res["weighted_sample_128x131072"] = {
            "draws_per_s": round(ph.shape[0] / t, 1), "s": round(t, 4),
            "exact_rows": int(np.sum(gw == rw)), "rows": int(ph.shape[0]),
            "matches_gpu_within_band": bool(all(band))}
        for kq, (tv, ti) in outputs["topk"].items():
            t, (rv, ri) = timed(lambda: oracle.topk_rows_f32(ph, kq), reps=1)
            res[f"topk_k{kq}_128x131072"] = {
                "rows_per_s": round(ph.shape[0] / t, 1), "s": round(t, 3),
                "matches_gpu": bool(np.array_equal(ti.cpu().numpy(), ri) and np.array_equal(
                    tv.cpu().numpy().view(np.uint32), rv.view(np.uint32)))}
    if "radix_keys" in outputs:
        kh = outputs["radix_keys"]
        sample = kh[: 1 << 22]
        t, _ = timed(lambda: oracle.sort_u32(sample), reps=1)
        rk, rp = oracle.sort_u32(kh)
        for bits in (8, 4, 1):
            ko, po = outputs[f"radix{bits}"]
            res[f"radix{bits}_n2^26"] = {
                "mkeys_per_s": round(sample.size / t / 1e6, 2),
                "sample": "first 2^22 keys of the workload (qsort of (key, index) pairs)",
                "matches_gpu": bool(np.array_equal(ko.cpu().numpy().view(np.uint32), rk) and
                                    np.array_equal(po.cpu().numpy(), rp))}
        kh16, ko16, po16 = outputs["radix_f16"]
        rk16, rp16 = oracle.sort_f16(kh16)
        res["radix8_f16_n2^26"] = {
            "matches_gpu": bool(np.array_equal(ko16.cpu().numpy().view(np.uint16),
                                               rk16.view(np.uint16)) and
                                np.array_equal(po16.cpu().numpy(), rp16))}
    return metric, res


if __name__ == "__main__":
    sys.exit(main())
