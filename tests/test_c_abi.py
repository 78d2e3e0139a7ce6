"""The C ABI from a C program: tests/c_abi/roundtrip.c is built with gcc
against include/bevpool.h, libbevpool.so and the oracle's C library, and run
as a child process (plan bit-exact against the oracle's cell map, pooled map
within 1e-4 sqrt(points per cell), documented error codes)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi", "roundtrip.c")
LIBDIR = os.path.join(ROOT, "paper_2205_13542_amd")
ROCM = "/opt/rocm"


def _build(tmp_path, oracle_dir):
    exe = str(tmp_path / "roundtrip")
    cmd = ["gcc", "-std=c11", "-O1", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           SRC, "-o", exe,
           "-L", LIBDIR, "-lbevpool", "-L", oracle_dir, "-loracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath," + LIBDIR, "-Wl,-rpath," + oracle_dir,
           "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    return exe


def test_c_program_builds(tmp_path, oracle_lib):
    """Header, library and oracle link from plain C (no GPU needed)."""
    if not os.path.exists(os.path.join(LIBDIR, "libbevpool.so")):
        pytest.skip("libbevpool.so is not built")
    _build(tmp_path, os.path.dirname(oracle_lib.LIB_PATH))


@pytest.mark.gpu
def test_c_roundtrip_on_gpu(tmp_path, oracle_lib):
    exe = _build(tmp_path, os.path.dirname(oracle_lib.LIB_PATH))
    print("[c roundtrip] running", flush=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("PASS"), r.stdout
