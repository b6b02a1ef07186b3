"""Build the gfx950 HIP library libdlm.so in-tree with hipcc."""

from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libdlm.so")
BUILD = os.path.join(HERE, "_build")
SOURCES = ["init.hip", "gemm.hip", "attention.hip", "elementwise.hip", "moe.hip", "engine.hip"]
ARCH = os.environ.get("DLM_OFFLOAD_ARCH", "gfx950")

CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 VALU forms are kept out of generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if c and (os.path.sep not in c or os.path.exists(c)):
            return c
    raise RuntimeError("hipcc not found")


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, src.replace(".hip", ".o"))
    cmd = [_hipcc(), *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def _device_asm(src: str) -> str:
    """gfx950 assembly of one source (kept for the static checks in tests/)."""
    asm = os.path.join(BUILD, src.replace(".hip", ".s"))
    cmd = [_hipcc(), *CFLAGS, "--cuda-device-only", "-S", os.path.join(CSRC, src), "-o", asm]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc -S failed for {src}:\n{r.stderr}")
    return asm


def build(jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(2 * len(SOURCES), os.cpu_count() or 4)
    with ThreadPoolExecutor(max_workers=jobs) as ex:
        obj_f = [ex.submit(_compile, s) for s in SOURCES]
        asm_f = [ex.submit(_device_asm, s) for s in SOURCES]
        objs = [f.result() for f in obj_f]
        for f in asm_f:
            f.result()
    tmp = OUT + f".tmp{os.getpid()}"
    cmd = [_hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, OUT)
    return OUT


# Host-code sanitizers: each flag goes to the host compilation only.
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer"]


def _clangxx() -> str:
    for c in (os.path.join(os.path.dirname(os.path.realpath(_hipcc())), "..", "llvm", "bin", "clang++"),
              "/opt/rocm/llvm/bin/clang++"):
        if os.path.exists(c):
            return os.path.realpath(c)
    raise RuntimeError("clang++ of the ROCm toolchain not found")


def build_host_sanitized() -> str:
    """The library with the host code of its C ABI (engine.hip: argument
    validation, planning, error paths) under AddressSanitizer and
    UndefinedBehaviorSanitizer; the kernel sources' objects are those of
    build(), and device code is never instrumented.  For CPU checks of the
    host paths: load it in a process that preloads the ASan runtime
    (asan_runtime())."""
    out_dir = os.path.join(BUILD, "hostsan")
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for src in SOURCES:
        if src != "engine.hip":
            obj = os.path.join(BUILD, src.replace(".hip", ".o"))
            if not os.path.exists(obj):
                _compile(src)
            objs.append(obj)
    obj = os.path.join(out_dir, "engine.o")
    cmd = [_hipcc(), *CFLAGS, *SANITIZE, "-c", os.path.join(CSRC, "engine.hip"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized host build failed:\n{r.stderr}")
    objs.append(obj)
    out = os.path.join(out_dir, "libdlm_hostsan.so")
    rocm = os.path.realpath(os.path.join(os.path.dirname(os.path.realpath(_hipcc())), ".."))
    # The sanitizer runtime is not linked in: the loading process preloads it,
    # and it resolves the objects' instrumentation calls.
    cmd = [_clangxx(), "-shared", "-fPIC", *objs, "-L" + os.path.join(rocm, "lib"), "-lamdhip64",
           "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized host link failed:\n{r.stderr}")
    return out


def asan_runtime() -> str:
    """Path of the toolchain's shared ASan runtime (to preload)."""
    r = subprocess.run([_clangxx(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    if r.returncode != 0 or not os.path.exists(path):
        raise RuntimeError("ASan runtime not found")
    return path


if __name__ == "__main__":
    print(build())
    sys.exit(0)
