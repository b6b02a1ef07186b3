"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The C ABI's host code (engine.hip: validation, planning, error paths, the
injected allocation failures) is rebuilt with both sanitizers and exercised
in a child process that preloads the toolchain's ASan runtime; the oracle's C
generator likewise, built with gcc.  Any sanitizer report ends the child with
a non-zero status.  No GPU work is launched: device code is never
instrumented, and the checks stop every call before a kernel launch.
"""

from __future__ import annotations

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CHECKS = os.path.join(ROOT, "tests", "host_checks.py")
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:abort_on_error=0:exitcode=23",
           "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _run(preload: str, *args: str) -> None:
    env = dict(os.environ, LD_PRELOAD=preload, **SAN_ENV)
    r = subprocess.run([sys.executable, CHECKS, *args], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0 and "host checks passed" in r.stdout, (r.returncode, r.stdout[-2000:],
                                                                    r.stderr[-6000:])


def test_c_abi_host_paths_under_asan_and_ubsan():
    import paper_2608_02625_amd.build as b
    lib = b.build_host_sanitized()
    _run(b.asan_runtime(), "abi", lib)


def test_oracle_generator_under_asan_and_ubsan():
    import oracle.build as ob
    lib, rt = ob.build_sanitized(os.path.join(ROOT, "paper_2608_02625_amd", "_build", "hostsan"))
    _run(rt, "oracle", lib, os.path.join(ROOT, "tests", "golden", "philox4x32_10_kat.txt"))
