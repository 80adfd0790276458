"""CPU builds under AddressSanitizer and UndefinedBehaviorSanitizer (no
GPU): the oracle's C sources driven through every entry point on heap
buffers of exactly their contract's sizes (tests/csrc/oracle_asan_main.c),
and the C-ABI's host code (abi.hip compiled for the host alone, its kernel
launchers replaced by recording stubs, tests/csrc/abi_stubs.cpp) driven
through every entry point with refused and accepted arguments, absurd
sizes included (tests/csrc/abi_host_main.cpp).  Any out-of-bounds access,
signed overflow or other undefined behaviour aborts the run."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]


def build_and_run(cmd, exe):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        if "asan" in r.stderr and ("cannot find" in r.stderr or "not found" in r.stderr):
            pytest.skip("no sanitizer runtime for this compiler")
        raise AssertionError("build failed:\n" + r.stderr[-3000:])
    env = dict(os.environ, ASAN_OPTIONS="halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    print(r.stdout)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    assert "0 failures" in r.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_asan")
    srcs = [os.path.join(ROOT, "oracle", f) for f in sorted(os.listdir(os.path.join(ROOT, "oracle")))
            if f.endswith(".c")]
    cmd = (["gcc", "-std=gnu11", "-ffp-contract=off", "-fno-fast-math"] + SAN +
           ["-I", os.path.join(ROOT, "oracle"), os.path.join(CSRC, "oracle_asan_main.c")] + srcs +
           ["-lm", "-o", exe])
    build_and_run(cmd, exe)


def test_abi_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_host")
    cmd = (["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__"] + SAN +
           ["-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
            "-I", os.path.join(ROOT, "paper_2609_22870_amd", "csrc"),
            "-x", "c++", os.path.join(ROOT, "paper_2609_22870_amd", "csrc", "abi.hip"), "-x", "none",
            os.path.join(CSRC, "abi_stubs.cpp"), os.path.join(CSRC, "abi_host_main.cpp"), "-o", exe])
    build_and_run(cmd, exe)
