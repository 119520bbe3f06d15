"""Register budget of the HIP kernels (CPU only: cross-compiles for gfx950).

A tile kernel keeps its tile in registers from its loads to its stores, so the
bytes in flight per CU -- and with them the bandwidth -- are set by how many
workgroups fit a CU.  Every tile kernel is built for at least 4 waves per SIMD
(at most 128 VGPRs: 16 waves per CU), and no kernel may spill
vector registers or use scratch memory (a spill adds private-segment traffic
and makes the runtime reserve scratch for every wave).  Scalar registers
spilled into vector-register lanes (the radix ranking keeps many 64-bit
ballot masks) touch no memory and are allowed.  This compiles each source to
device assembly and reads the resource metadata the compiler emits for every
kernel.
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2505_15112_amd import build as B

SOURCES = sorted(f for f in os.listdir(B.CSRC) if f.endswith(".hip"))
TILE_KERNELS = ("k_scan_lookback", "k_scan_lookback_lds", "k_scan_mfma_f16", "k_rss_reduce",
                "k_rss_rescan", "k_rows_lookback", "k_topp", "k_topp_head", "k_topp_finish", "k_compact",
                "k_split", "k_radix4_count", "k_radix4_scatter", "k_radix8_count", "k_topk_gather",
                "k_radix8_scatter", "k_topk_hist", "k_topk_select")


def test_lds_tile_workgroup_fits_a_cu(tmp_path):
    """The register + LDS scan tile (one 16-wave workgroup per CU) must fit
    the CU's 160 KB of LDS."""
    src = os.path.join(B.CSRC, "scan1d.hip")
    out = tmp_path / "scan1d.s"
    flags = [f for f in B.CFLAGS if f != "-fPIC"]
    subprocess.run([B.HIPCC, *flags, "--cuda-device-only", "-S", src, "-o", str(out)],
                   check=True, capture_output=True)
    meta = out.read_text()
    meta = meta[meta.index("amdhsa.kernels"):]
    sizes = []
    for block in meta.split("  - .agpr_count")[1:]:
        name = re.search(r"\.name:\s+(\S+)", block).group(1)
        if "k_scan_lookback_lds" in name:
            sizes.append(int(re.search(r"\.group_segment_fixed_size:\s+(\d+)", block).group(1)))
    assert sizes and max(sizes) <= 160 * 1024, sizes


@pytest.mark.skipif(shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC),
                    reason="hipcc not available")
def test_topk_tile_kernels_fit_eight_waves(tmp_path):
    """The top-k tile kernels that keep candidates (4-wave workgroups, each
    holding 8192 keys in registers) are sized so that 8 workgroups share a
    CU: at most 64 VGPRs and 20 KB of LDS each, which keeps all 2048 tiles of
    a 128 x 131072 call resident at once."""
    src = os.path.join(B.CSRC, "topk.hip")
    out = tmp_path / "topk.s"
    flags = [f for f in B.CFLAGS if f != "-fPIC"]
    subprocess.run([B.HIPCC, *flags, "--cuda-device-only", "-S", src, "-o", str(out)],
                   check=True, capture_output=True)
    meta = out.read_text()
    meta = meta[meta.index("amdhsa.kernels"):]
    seen = 0
    for block in meta.split("  - .agpr_count")[1:]:
        name = re.search(r"\.name:\s+(\S+)", block).group(1)
        if "k_topk_tilesel" in name or "k_topk_gather" in name:
            seen += 1
            vgpr = int(re.search(r"\.vgpr_count:\s+(\d+)", block).group(1))
            lds = int(re.search(r"\.group_segment_fixed_size:\s+(\d+)", block).group(1))
            assert vgpr <= 64 and lds * 8 <= 160 * 1024, (name, vgpr, lds)
    assert seen


def kernel_resources(src, tmp_path):
    out = tmp_path / (os.path.basename(src) + ".s")
    flags = [f for f in B.CFLAGS if f != "-fPIC"]
    subprocess.run([B.HIPCC, *flags, "--cuda-device-only", "-S", src, "-o", str(out)],
                   check=True, capture_output=True)
    text = out.read_text()
    meta = text[text.index("amdhsa.kernels"):]
    res = {}
    for block in meta.split("  - .agpr_count")[1:]:
        def field(key):
            m = re.search(r"\." + key + r":\s+(\S+)", block)
            return m.group(1) if m else None
        res[field("name")] = {k: int(field(k) or 0) for k in (
            "vgpr_count", "sgpr_count", "vgpr_spill_count", "sgpr_spill_count",
            "private_segment_fixed_size")}
    return res


@pytest.mark.skipif(shutil.which(B.HIPCC) is None and not os.path.exists(B.HIPCC),
                    reason="hipcc not available")
@pytest.mark.parametrize("source", SOURCES)
def test_no_spills_and_tile_kernels_fit_128_vgprs(source, tmp_path):
    res = kernel_resources(os.path.join(B.CSRC, source), tmp_path)
    if not res:
        pytest.skip(f"{source} defines no kernels")
    bad = []
    for name, r in res.items():
        if r["vgpr_spill_count"] or r["private_segment_fixed_size"]:
            bad.append(f"{name}: spills/scratch {r}")
        if any(k in name for k in TILE_KERNELS) and r["vgpr_count"] > 128:
            bad.append(f"{name}: {r['vgpr_count']} VGPRs > 128")
    assert not bad, "\n".join(bad)
