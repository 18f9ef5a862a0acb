"""Compile tests/c/abi_roundtrip (a plain C program using include/mezo.h,
libmezo.so, the HIP runtime's C API and the oracle's C library). Test
infrastructure: called by __graft_entry__.build()."""
from __future__ import annotations

import subprocess
from pathlib import Path

HERE = Path(__file__).resolve().parent
ROOT = HERE.parent.parent
BIN = HERE / "abi_roundtrip"


def build() -> Path:
    pkg = ROOT / "paper_2306_10015_amd"
    cmd = ["gcc", "-std=c99", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", str(ROOT / "include"), "-I", str(ROOT / "oracle"), "-I", "/opt/rocm/include",
           str(HERE / "abi_roundtrip.c"), "-o", str(BIN),
           "-L", str(pkg), "-lmezo", "-L", str(ROOT / "oracle"), "-loracle",
           "-L", "/opt/rocm/lib", "-lamdhip64", "-lm",
           f"-Wl,-rpath,{pkg}", f"-Wl,-rpath,{ROOT / 'oracle'}", "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building {BIN.name} failed:\n{r.stderr}")
    return BIN


if __name__ == "__main__":
    print(build())
