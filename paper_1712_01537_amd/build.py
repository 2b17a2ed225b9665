"""Compile the HIP sources under csrc/ into liboc.so for gfx950 (in-tree)."""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import re
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "liboc.so")
OBJ = os.path.join(ROOT, "_build", "obj")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    # packed-FP32 instructions are kept out of every kernel on purpose
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]


# Kernels that wait on a compile-time count of outstanding vector-memory
# operations (inline "s_waitcnt vmcnt(N)") are only correct when the compiler
# adds no memory operations of its own to the count: a register spill to
# scratch memory does, and would let an LDS read race the DMA it waits for
# (wrong data, no error).  Every kernel of a source file that holds such a wait
# must therefore use no scratch memory; the compiler's resource-usage remarks
# are checked after each compile and the build fails otherwise.
COUNTED_WAIT = re.compile(r"s_waitcnt vmcnt\(%")


def _scratch_by_kernel(remarks: str) -> dict:
    """Kernel (mangled name) -> scratch bytes per lane, from the compiler's
    -Rpass-analysis=kernel-resource-usage remarks."""
    out, name = {}, None
    for ln in remarks.splitlines():
        m = re.search(r"remark: Function Name: (\S+)", ln)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"remark:\s+ScratchSize \[bytes/lane\]: (\d+)", ln)
        if m and name:
            out[name] = int(m.group(1))
    return out


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.basename(src) + ".o")
    cmd = [HIPCC, *FLAGS, "-Rpass-analysis=kernel-resource-usage", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    with open(src) as fh:
        counted = COUNTED_WAIT.search(fh.read()) is not None
    if counted:
        bad = {k: v for k, v in _scratch_by_kernel(r.stderr).items() if v > 0}
        if bad:
            os.remove(obj)
            raise RuntimeError(f"{src} holds counted vmcnt waits, but these kernels use scratch "
                               f"memory (bytes/lane), which breaks the counts: {bad}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(OBJ, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
