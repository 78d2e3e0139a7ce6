"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only,
no GPU): the CPU oracle run through every function on small rigs, and the C
ABI's host layer (argument checks, messages, plan ownership) run through its
error paths with the device work and HIP runtime calls stubbed. Any
out-of-bounds access, use after free, leak, signed overflow or bad shift
aborts the program and fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CABI = os.path.join(ROOT, "tests", "c_abi")
CSRC = os.path.join(ROOT, "paper_2205_13542_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", OMP_NUM_THREADS="2")


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=ENV)
    assert r.returncode == 0 and r.stdout.strip().endswith("PASS"), r.stdout + r.stderr


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_sanitize")
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fopenmp",
           os.path.join(CABI, "oracle_sanitize.c"), os.path.join(ROOT, "oracle", "bevpool_oracle.c"),
           "-o", exe, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    _run(exe)


@pytest.mark.skipif(not os.path.exists(HIPCC) and not shutil.which("hipcc"), reason="no hipcc")
def test_abi_host_layer_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_host_sanitize")
    # host pass only, sanitizers for the host code (no device code is built)
    cmd = [HIPCC, "-std=c++17", "--offload-arch=gfx950", "--cuda-host-only", "-O1", "-g",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-fno-gpu-sanitize", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "bevpool.hip"), os.path.join(CABI, "abi_host_sanitize.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr
    _run(exe)
