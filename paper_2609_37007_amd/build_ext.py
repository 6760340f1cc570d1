"""Build librvqsd.so (HIP kernels + host runtime) in-tree for gfx950.

Each source compiles to its own object in a temporary folder, in parallel,
then one link step writes the shared library."""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "librvqsd.so")
SOURCES = [os.path.join(CSRC, "rvqsd_frame.hip"), os.path.join(CSRC, "rvqsd_batch.hip"),
           os.path.join(CSRC, "rvqsd_noalloc.hip"), os.path.join(CSRC, "rvqsd_api.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# packed FP32 instructions are disabled for all device code
FLAGS = ["-O3", "--offload-arch=gfx950", "-std=c++17", "-fPIC", "-Wall",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
NOISE = "is not a recognized feature for this target"


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    msg = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if NOISE not in l)
    return r.returncode, msg


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory(prefix="rvqsd_build_") as d:
        objs = [os.path.join(d, os.path.basename(src) + ".o") for src in SOURCES]
        cmds = [[HIPCC] + FLAGS + ["-c", src, "-o", obj] for src, obj in zip(SOURCES, objs)]
        with cf.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            results = list(ex.map(_run, cmds))
        for cmd, (rc, msg) in zip(cmds, results):
            if verbose:
                print(" ".join(cmd), flush=True)
            if rc != 0:
                raise RuntimeError(f"hipcc failed ({rc}):\n{msg}")
            if verbose and msg.strip():
                print(msg)
        link = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + objs + ["-o", tmp]
        rc, msg = _run(link)
        if verbose:
            print(" ".join(link), flush=True)
        if rc != 0:
            raise RuntimeError(f"link failed ({rc}):\n{msg}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
