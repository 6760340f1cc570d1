"""Build librvqsd.so (HIP kernels + host runtime) in-tree for gfx950.

Each source compiles to its own object in a temporary folder, in parallel,
then one link step writes the shared library. Alongside, the device code of
every HIP source is compiled to assembly and checked: no instruction may read
a register that an inline-assembly device-coherent load (pload4) is still
filling, i.e. before the s_waitcnt vmcnt(0) of its vm_wait. The compiler does
not know that such a load is outstanding and may copy its destination early
under register pressure; the build fails if it does."""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
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


_KERNEL = re.compile(r"^(_Z\S+):")
_COH_LOAD = re.compile(r"global_load_dwordx4 v\[(\d+):(\d+)\], v\[\d+:\d+\], off sc1")
_RANGE = re.compile(r"\bv\[(\d+):(\d+)\]")
_REG = re.compile(r"\bv(\d+)\b")


def inflight_reads(asm: str) -> list:
    """(kernel, line) of every instruction that reads or writes a VGPR of an
    inline-assembly coherent 16-byte load before the next s_waitcnt vmcnt(0),
    scanning each function's instructions in layout order."""
    found, kern, pending = [], None, set()
    for line in asm.splitlines():
        m = _KERNEL.match(line)
        if m:
            kern, pending = m.group(1), set()
            continue
        s = line.split(";")[0].strip()
        if kern is None or not s or s.startswith(".") or s.endswith(":"):
            continue
        m = _COH_LOAD.search(s)
        if m:
            pending.update(range(int(m.group(1)), int(m.group(2)) + 1))
            continue
        if "s_waitcnt" in s and "vmcnt(0)" in s or s.startswith(("s_endpgm", "s_setpc", "s_swappc")):
            pending = set()
            continue
        if pending:
            regs = {r for a, b in _RANGE.findall(s) for r in range(int(a), int(b) + 1)}
            regs.update(int(r) for r in _REG.findall(s))
            if regs & pending:
                found.append((kern, s))
    return found


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory(prefix="rvqsd_build_") as d:
        objs = [os.path.join(d, os.path.basename(src) + ".o") for src in SOURCES]
        cmds = [[HIPCC] + FLAGS + ["-c", src, "-o", obj] for src, obj in zip(SOURCES, objs)]
        hips = [src for src in SOURCES if src.endswith(".hip")]
        asms = [os.path.join(d, os.path.basename(src) + ".s") for src in hips]
        cmds += [[HIPCC] + FLAGS + ["--cuda-device-only", "-S", src, "-o", s] for src, s in zip(hips, asms)]
        with cf.ThreadPoolExecutor(max_workers=len(cmds)) as ex:
            results = list(ex.map(_run, cmds))
        for cmd, (rc, msg) in zip(cmds, results):
            if verbose:
                print(" ".join(cmd), flush=True)
            if rc != 0:
                raise RuntimeError(f"hipcc failed ({rc}):\n{msg}")
            if verbose and msg.strip():
                print(msg)
        for src, s in zip(hips, asms):
            with open(s) as f:
                bad = inflight_reads(f.read())
            if bad:
                shown = "\n".join(f"  {k}: {i}" for k, i in bad[:8])
                raise RuntimeError(f"{os.path.basename(src)}: {len(bad)} instruction(s) touch the destination of an "
                                   f"unfinished coherent load:\n{shown}")
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
