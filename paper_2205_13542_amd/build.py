"""Build libbevpool.so for gfx950 with hipcc, in-tree.

``python -m paper_2205_13542_amd.build`` (or ``build()``) always recompiles,
so a stale library never survives a source change.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB_PATH = os.path.join(HERE, "libbevpool.so")
# measurement probe for bench.py --floor (not part of the pooling library)
FLOOR_SOURCE = "floor.hip"
FLOOR_LIB_PATH = os.path.join(HERE, "libbevpool_floor.so")
SOURCES = ["bevpool.hip", "plan.hip", "forward.hip", "backward.hip", "layout.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC", "-shared",
    # bit-exact plan geometry: no contraction into fused multiply-adds
    "-ffp-contract=off",
    # no packed fp32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-fvisibility=hidden",
]


def build(verbose: bool = False) -> str:
    """Compile every source to an object in parallel, then link the library."""
    import concurrent.futures
    import tempfile
    compile_flags = [f for f in FLAGS if f != "-shared"]
    with tempfile.TemporaryDirectory(prefix="bevpool_build_") as tmpdir:
        objs = [os.path.join(tmpdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
        cmds = [[HIPCC, *compile_flags, "-I", INCLUDE, "-I", CSRC, "-c",
                 os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
        floor_tmp = FLOOR_LIB_PATH + ".tmp"
        cmds.append([HIPCC, *FLAGS, os.path.join(CSRC, FLOOR_SOURCE), "-o", floor_tmp])
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        workers = max(1, min(len(cmds), os.cpu_count() or 1))
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            for r in ex.map(lambda c: subprocess.run(c, capture_output=True, text=True), cmds):
                if r.returncode != 0:
                    raise subprocess.CalledProcessError(r.returncode, r.args, r.stdout, r.stderr)
        tmp = LIB_PATH + ".tmp"
        subprocess.run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp],
                       check=True)
        os.replace(floor_tmp, FLOOR_LIB_PATH)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
