"""Build libgsmi.so (gfx950) in-tree with hipcc.

Every kernel file is compiled with packed-FP32 instructions disabled
(-Xclang -target-feature -Xclang -packed-fp32-ops); the projection file is
also built with -ffp-contract=off because its fp32 geometry must follow a
fixed operation order, the optimizer file because a parameter must
change by exactly the step it publishes (no fused multiply-add), and the
host planner because its doubles follow a fixed operation order.  Usage:  python -m paper_2607_19893_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libgsmi.so")
BUILD_DIR = os.path.join(os.path.dirname(HERE), "_build", "gsmi")
ARCH = os.environ.get("GSMI_ARCH", "gfx950")

SOURCES = ["project.hip", "compact.hip", "binsort.hip", "raster.hip", "adam.hip", "delta.hip", "scope.hip",
           "planner.cpp", "abi.cpp"]
STRICT_FP = {"project.hip", "adam.hip", "planner.cpp"}


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _flags(src: str):
    f = ["-O3", "-fPIC", "-std=c++17", "--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops", "-Wno-unused-command-line-argument", "-I" + os.path.join(os.path.dirname(HERE), "include")]
    if src in STRICT_FP:
        f.append("-ffp-contract=off")
    if src.endswith(".cpp"):
        f += ["-x", "hip"]
    return f


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, src + ".o")
    cmd = [hipcc()] + _flags(src) + ["-Rpass-analysis=kernel-resource-usage", "-c", os.path.join(CSRC, src),
                                     "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr[-6000:]))
    check_no_scratch(src, r.stderr)
    return obj


def check_no_scratch(src: str, remarks: str) -> None:
    """Refuse kernels that use private (scratch) memory: besides the slow
    memory path, a launch that needs scratch can stall the launching thread
    while the runtime sets scratch up for the queue, which showed up as gaps
    of up to 43 ms between kernels of a training step."""
    name = None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and int(m.group(1)) > 0:
            raise RuntimeError("%s: kernel %s uses %s bytes of scratch per lane" % (src, name, m.group(1)))


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4)))
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = OUT + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "-shared", "-fPIC", "--offload-arch=" + ARCH, "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr[-4000:]))
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
