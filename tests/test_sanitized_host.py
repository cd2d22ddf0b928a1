"""The loader and the oracle under AddressSanitizer and UBSan (CPU only).

Builds echo_host.cpp (validation, matching, levelling, walk lists, upload,
walk-chain analysis) with g++ -fsanitize=address,undefined, linked against a
host-memory stand-in of the HIP runtime (tests/sanitize/hip_host_stub.cpp), and
the oracle (oracle/echo_oracle.c) with gcc and the same sanitizers; then runs
the ABI tests, the oracle pins and the stub-only loader tests (forced
allocation failures, walk-chain hand cases) against those builds in a child
pytest, with the AddressSanitizer runtime preloaded into it.  Any report
(out-of-bounds access, use after free, undefined behaviour) fails the run.
"""
from __future__ import annotations

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined"]


def _asan_runtime():
    try:
        p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True,
                           check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        return None
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    if os.environ.get("LD_PRELOAD"):
        pytest.skip("another library is preloaded; the AddressSanitizer runtime must come first")
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("gcc's AddressSanitizer runtime is not installed")
    out = tmp_path_factory.mktemp("sanitize")
    host = str(out / "libecho_host_san.so")
    orc = str(out / "liboracle_san.so")
    csrc = os.path.join(ROOT, "paper_2412_12487_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", *SAN, "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__",
                    "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"), "-I", csrc,
                    os.path.join(csrc, "echo_host.cpp"), os.path.join(ROOT, "tests", "sanitize", "hip_host_stub.cpp"),
                    "-o", host], check=True)
    subprocess.run(["gcc", "-std=c11", *SAN, "-fPIC", "-shared", "-pthread",
                    os.path.join(ROOT, "oracle", "echo_oracle.c"), "-o", orc], check=True)
    return {"runtime": rt, "host": host, "oracle": orc}


def test_loader_and_oracle_under_sanitizers(sanitized):
    env = dict(os.environ)
    env.update(LD_PRELOAD=sanitized["runtime"], ECHO_SANITIZED_LIB=sanitized["host"],
               ORACLE_SANITIZED_LIB=sanitized["oracle"], ECHO_HOST_STUB="1",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        "-p", "tests.sanitize.plugin", "-m", "not gpu",
                        "tests/test_abi.py", "tests/test_oracle_pins.py", "tests/sanitize/test_stubbed_loader.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=1500)
    tail = (r.stdout[-6000:] + "\n" + r.stderr[-6000:])
    assert r.returncode == 0, tail
    assert " passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail
