"""Build the oracle's C part (the weight generator) with gcc.

CPU oracle -- test infrastructure only.
"""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "rng.c")
LIB = os.path.join(HERE, "_oracle_rng.so")


def build(force: bool = True) -> str:
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_sanitized(out_dir: str) -> tuple[str, str]:
    """The same C under AddressSanitizer and UndefinedBehaviorSanitizer (gcc,
    host code only, OpenMP off), for CPU checks; returns (library, the ASan
    runtime a process loading it must preload)."""
    os.makedirs(out_dir, exist_ok=True)
    lib = os.path.join(out_dir, "liboracle_rng_san.so")
    cmd = ["gcc", "-O1", "-g", "-fPIC", "-shared", "-std=c99", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", SRC, "-o", lib]
    subprocess.run(cmd, check=True)
    rt = subprocess.run(["gcc", "-print-file-name=libasan.so"], check=True, capture_output=True,
                        text=True).stdout.strip()
    return lib, os.path.realpath(rt)


if __name__ == "__main__":
    print(build())
