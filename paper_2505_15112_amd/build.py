"""Build libscan.so (the HIP kernels and the C ABI) for gfx950 with hipcc.

    python -m paper_2505_15112_amd.build [-v]

Compiles every csrc/*.hip into _build/ and links paper_2505_15112_amd/libscan.so
in-tree.  Always recompiles.  Also links libscan_adv.so, the same sources built
with LS_ADVERSARIAL_DELAYS (pseudo-random pauses before every inter-workgroup
protocol step) for the adversarial-scheduling tests; it binds its own symbols
(-Bsymbolic) so that it can be loaded beside libscan.so.
"""
import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build", "libscan")
LIB = os.path.join(PKG, "libscan.so")
LIB_ADV = os.path.join(PKG, "libscan_adv.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra",
    "-Wno-unused-parameter",
    # Packed-FP32 instructions stay off (they are not needed by any kernel here).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-mcode-object-version=5",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str, verbose: bool, build_dir: str, extra=()) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, *extra, "-c", src, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l
                     and "not a recognized feature" not in l and l.strip())
    if warn and verbose:
        print(warn, file=sys.stderr)
    return obj


def _link(objs, out: str, verbose: bool, extra=()) -> str:
    tmp = out + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *extra, "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> str:
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    adv_dir = BUILD + "_adv"
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(adv_dir, exist_ok=True)
    jobs = [(s, BUILD, ()) for s in srcs] + [(s, adv_dir, ("-DLS_ADVERSARIAL_DELAYS",)) for s in srcs]
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        objs = list(ex.map(lambda j: _compile(j[0], verbose, j[1], j[2]), jobs))
    _link(objs[:len(srcs)], LIB, verbose)
    _link(objs[len(srcs):], LIB_ADV, verbose, ("-Wl,-Bsymbolic",))
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
