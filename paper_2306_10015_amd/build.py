"""Compile libmezo.so (the HIP kernels for gfx950 plus the C ABI) in-tree.

    python -m paper_2306_10015_amd.build

Flags that fix the arithmetic: -ffp-contract=off (only the fma the source
writes is fused), no fast-math, correctly rounded fp32 / and sqrt (the
portable Gaussian relies on them), and packed fp32 instructions disabled.
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
CSRC = PKG / "csrc"
ROOT = PKG.parent
LIB = PKG / "libmezo.so"
PROBE_LIB = PKG / "libstream_probe.so"
BUILD_DIR = ROOT / "_build"

ARCH = "gfx950"
COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wextra", "-ffp-contract=off",
          "-I" + str(ROOT / "include"), "-I" + str(CSRC)]
# Code object v5: loadable by the HIP runtime that ships with PyTorch as well
# as by the system one.
DEVICE = ["--offload-arch=" + ARCH, "-mcode-object-version=5",
          "-fhip-fp32-correctly-rounded-divide-sqrt",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd) -> list[str]:
    """Run a compiler command; returns its kernel resource remarks."""
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass reports the device-only feature flag as unknown: harmless
    noise = "'-packed-fp32-ops' is not a recognized feature"
    lines = [l for l in r.stderr.splitlines() if noise not in l]
    remarks = [l for l in lines if RESOURCE_REMARK in l]
    # the remarks' source excerpts ("  42 | {", "     | ^") go with them
    err = "\n".join(l for l in lines if RESOURCE_REMARK not in l and not _EXCERPT.match(l))
    if r.returncode != 0:
        raise RuntimeError(f"command failed: {' '.join(cmd)}\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return remarks


RESOURCE_REMARK = "-Rpass-analysis=kernel-resource-usage"
_EXCERPT = re.compile(r"^\s*\d*\s*\|")
_REMARK_FIELD = re.compile(r"remark:\s+([A-Za-z ]+?)(?: \[[^]]*\])?:\s+(\S+)")


def kernel_resources(remarks: list[str]) -> list[dict]:
    """One entry per kernel from the compiler's resource-usage remarks: its
    name, VGPRs, scratch bytes per lane and occupancy (waves per SIMD)."""
    out: list[dict] = []
    for line in remarks:
        m = _REMARK_FIELD.search(line)
        if not m:
            continue
        key, val = m.group(1).strip(), m.group(2)
        if key == "Function Name":
            out.append({"kernel": val})
        elif out and key in ("VGPRs", "ScratchSize", "Occupancy"):
            out[-1][key] = int(val)
    return out


#: The kernel translation units of libmezo, one object each.
KERNEL_UNITS = ["engine_dense.hip", "engine_nf4.hip", "nf4_convert.hip", "checksum.hip", "inspect.hip",
                "noalloc.hip"]


def build(verbose: bool = False) -> Path:
    """Compile the kernel units and api.cpp and link libmezo.so next to this
    file; compile the streaming probe the benchmark measures against into
    libstream_probe.so."""
    BUILD_DIR.mkdir(exist_ok=True)
    cc = hipcc()
    objs = []
    table = []
    for unit in KERNEL_UNITS:
        obj = BUILD_DIR / (Path(unit).stem + ".o")
        remarks = _run([cc, *COMMON, *DEVICE, RESOURCE_REMARK, "-c", str(CSRC / unit), "-o", str(obj)])
        table += [dict(unit=unit, **k) for k in kernel_resources(remarks)]
        objs.append(str(obj))
    # every kernel keeps its values in registers: a spill to per-lane scratch
    # memory is a build error
    with open(BUILD_DIR / "kernel_resources.txt", "w") as f:
        for k in table:
            f.write(f"{k['unit']} {k['kernel']} vgprs={k.get('VGPRs')} scratch={k.get('ScratchSize')} "
                    f"waves_per_simd={k.get('Occupancy')}\n")
    spills = [k for k in table if k.get("ScratchSize", 0) > 0]
    if not table or spills:
        raise RuntimeError("kernels using scratch memory: "
                           + (", ".join(k["kernel"] for k in spills) if table else "(no resource remarks)"))
    a_obj = BUILD_DIR / "api.o"
    _run([cc, *COMMON, "-c", str(CSRC / "api.cpp"), "-o", str(a_obj)])
    tmp = LIB.with_suffix(".so.tmp")
    _run([cc, "-shared", "-fPIC", *DEVICE, *objs, str(a_obj), "-o", str(tmp)])
    os.replace(tmp, LIB)
    # the benchmark's streaming ceiling probe (measurement only, not part of libmezo)
    ptmp = PROBE_LIB.with_suffix(".so.tmp")
    _run([cc, *COMMON, *DEVICE, "-shared", str(CSRC / "stream_probe.hip"), "-o", str(ptmp)])
    os.replace(ptmp, PROBE_LIB)
    if verbose:
        print(f"built {LIB} and {PROBE_LIB.name}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
