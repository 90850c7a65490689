"""Build libdsmpnn.so (gfx950) in-tree with hipcc.

Every HIP source is compiled for gfx950 only, with packed-FP32 instructions
disabled, and linked into one shared library next to this file
(``lib/libdsmpnn.so``).  The radius-graph source is compiled with
floating-point contraction off so the distance test keeps its roundings.

The build fails if any kernel uses scratch memory (register spills):
several kernels wait for their own copies with explicit vector-memory counts,
and scratch loads and stores would count among them.
"""

import os
import re
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "lib")
LIB = os.path.join(OUT_DIR, "libdsmpnn.so")
BUILD_DIR = os.path.join(HERE, "_build")

SOURCES = ["core.hip", "graph.hip", "nnconv_fwd.hip", "nnconv_bwd.hip", "nnconv_agg.hip", "hop.hip"]
COMMON = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
PER_FILE = {"graph.hip": ["-ffp-contract=off"]}


def _hipcc():
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def scratch_kernels(remarks: str):
    """Kernels that the compiler's resource-usage remarks show with a nonzero
    scratch size."""
    out, name = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
            continue
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name is not None and int(m.group(1)) > 0:
            out.append("%s (%s bytes/lane)" % (name, m.group(1)))
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    os.makedirs(BUILD_DIR, exist_ok=True)
    hipcc = _hipcc()

    def compile_one(src):
        obj = os.path.join(BUILD_DIR, src + ".o")
        cmd = [hipcc] + COMMON + PER_FILE.get(src, []) + ["-Rpass-analysis=kernel-resource-usage",
                                                           "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError("hipcc failed for %s:\n%s" % (src, r.stderr[-8000:]))
        spills = scratch_kernels(r.stderr)
        if spills:
            raise RuntimeError("kernels of %s use scratch memory: %s" % (src, ", ".join(spills)))
        if verbose:
            sys.stderr.write("".join(l + "\n" for l in r.stderr.splitlines() if "remark" not in l))
        return obj

    with ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s" % r.stderr[-8000:])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
