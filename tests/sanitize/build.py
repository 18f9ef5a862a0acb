"""Build the sanitized host check of the C ABI (CPU only; test infrastructure).

api.cpp and the HIP stand-in (hip_double.cpp) are compiled by g++, the driver
(abi_host_check.c) by gcc, all with AddressSanitizer and
UndefinedBehaviorSanitizer, into one program that needs no GPU and no HIP
runtime library: the stand-in defines every HIP call api.cpp makes.

    python tests/sanitize/build.py   ->  tests/sanitize/abi_host_check
"""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

HERE = Path(__file__).resolve().parent
ROOT = HERE.parent.parent
CSRC = ROOT / "paper_2306_10015_amd" / "csrc"
EXE = HERE / "abi_host_check"
BUILD = ROOT / "_build" / "sanitize"

SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]
INC = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT / 'include'}", f"-I{CSRC}"]


def build() -> Path:
    BUILD.mkdir(parents=True, exist_ok=True)
    objs = []
    for src, cc, std in [(CSRC / "api.cpp", "g++", "-std=c++17"), (HERE / "hip_double.cpp", "g++", "-std=c++17"),
                         (HERE / "abi_host_check.c", "gcc", "-std=c99")]:
        obj = BUILD / (src.stem + ".o")
        subprocess.run([cc, std, *SAN, *INC, "-Wall", "-Wextra", "-c", str(src), "-o", str(obj)], check=True)
        objs.append(str(obj))
    tmp = EXE.with_suffix(".tmp")
    subprocess.run(["g++", *SAN, *objs, "-o", str(tmp), "-lpthread", "-lm"], check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build())
    sys.exit(0)
