"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

oracle.c is rebuilt with -fsanitize=address,undefined (gcc, host code; no GPU
code is involved) and every pin of oracle_pins.py runs through that build in a
child Python whose first loaded libraries are the sanitizer runtimes.  An
out-of-bounds access, a use after free, signed overflow, a misaligned load or
an out-of-range shift anywhere in the oracle on the pins' inputs aborts the
child.  A control library with a planted one-element heap overflow must abort
the same way, which shows that the sanitizers are in effect in this setup.  The
C ABI's host code (argument validation in abi.hip) is built the same way --
each -fsanitize= after -Xarch_host, so no GPU code is instrumented -- and the
CPU ABI tests run against it.
"""
import os
import shutil
import subprocess
import sys
import textwrap

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_DIR = os.path.join(ROOT, "oracle")
SAN_FLAGS = ["-O1", "-g", "-std=c11", "-fPIC", "-shared", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


ASAN, UBSAN = _runtime("libasan.so"), _runtime("libubsan.so")
pytestmark = pytest.mark.skipif(shutil.which("gcc") is None or not ASAN or not UBSAN,
                                reason="gcc with the sanitizer runtimes is needed")

RUNNER = textwrap.dedent("""
    import sys
    sys.path[:0] = [{root!r}, {tests!r}]
    import oracle, oracle_pins as P
    o = oracle.Oracle(sys.argv[1])
    for check in P.ALL_CHECKS:
        check(o)
    print("PINS_OK", len(P.ALL_CHECKS))
""")


def _env():
    env = dict(os.environ)
    env["LD_PRELOAD"] = f"{ASAN}:{UBSAN}"
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    return env


def _build(src, out):
    subprocess.run(["gcc", *SAN_FLAGS, "-I", ORACLE_DIR, "-o", str(out), str(src), "-lm"],
                   check=True, capture_output=True)


def _run(lib, tmp_path):
    script = tmp_path / "run_pins.py"
    script.write_text(RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests")))
    return subprocess.run([sys.executable, str(script), str(lib)], env=_env(),
                          capture_output=True, text=True, timeout=600)


def test_every_pin_passes_under_asan_and_ubsan(tmp_path):
    lib = tmp_path / "liboracle_san.so"
    _build(os.path.join(ORACLE_DIR, "oracle.c"), lib)
    r = _run(lib, tmp_path)
    assert r.returncode == 0 and "PINS_OK" in r.stdout, (r.stdout[-2000:], r.stderr[-4000:])


def test_planted_overflow_is_caught(tmp_path):
    """Control: the oracle's inclusive int32 scan with its loop bound off by
    one (it writes y[n]) must abort under the same setup."""
    src = open(os.path.join(ORACLE_DIR, "oracle.c")).read()
    needle = "for (int64_t i = 0; i < n; ++i)"
    head, sep, tail = src.partition("oracle_scan_inclusive_i32")
    assert sep and needle in tail, "the scan loop this control edits has moved"
    planted = tmp_path / "oracle_planted.c"
    planted.write_text(head + sep + tail.replace(needle, "for (int64_t i = 0; i <= n; ++i)", 1))
    lib = tmp_path / "liboracle_planted.so"
    _build(planted, lib)
    r = _run(lib, tmp_path)
    assert r.returncode != 0 and "PINS_OK" not in r.stdout, r.stdout[-2000:]
    assert "AddressSanitizer" in r.stderr, r.stderr[-2000:]


ABI_RUNNER = textwrap.dedent("""
    import sys
    sys.path[:0] = [{root!r}, {tests!r}]
    from paper_2505_15112_amd import _lib
    _lib.load(sys.argv[1])  # every later _lib.load() returns this library
    assert sys.argv[1] in open("/proc/self/maps").read()
    import pytest
    sys.exit(pytest.main(["-q", "-x", "-p", "no:cacheprovider", {abi_tests!r}]))
""")


def test_abi_validation_under_asan_and_ubsan(tmp_path):
    """The C ABI's host-side argument checks (abi.hip, host code instrumented;
    its kernels are not) run every CPU ABI test without a sanitizer report.
    The other objects come from the regular build."""
    from paper_2505_15112_amd import build as B
    objs = sorted(os.path.join(B.BUILD, f) for f in os.listdir(B.BUILD)
                  if f.endswith(".hip.o") and f != "abi.hip.o") if os.path.isdir(B.BUILD) else []
    if not objs:
        pytest.skip("libscan objects not built (run the package build first)")
    host_san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-omit-frame-pointer"]
    flags = [f for f in B.CFLAGS if f != "-O3"] + ["-O1", "-g"]
    abi_o = tmp_path / "abi_san.o"
    subprocess.run([B.HIPCC, *flags, *host_san, "-c", os.path.join(B.CSRC, "abi.hip"), "-o",
                    str(abi_o)], check=True, capture_output=True)
    lib = tmp_path / "libscan_san.so"
    subprocess.run([B.HIPCC, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *host_san[:4], "-o",
                    str(lib), str(abi_o), *objs], check=True, capture_output=True)
    script = tmp_path / "run_abi.py"
    script.write_text(ABI_RUNNER.format(root=ROOT, tests=os.path.join(ROOT, "tests"),
                                        abi_tests=os.path.join(ROOT, "tests", "test_abi_cpu.py")))
    r = subprocess.run([sys.executable, str(script), str(lib)], env=_env(), capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
