"""Build libjpi.so (HIP, gfx950) in-tree, plus the seeded input generator."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libjpi.so")
SOURCES = ["jpi_kernels.hip", "jpi_flash.hip", "jpi_block.hip", "jpi_variant.hip", "jpi_persist.hip", "jpi_runtime.hip", "jpi_vlm.hip", "jpi_corr.hip", "jpi_noalloc.hip", "jpi_sched.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         # no packed-fp32 instructions in device code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        sys.stderr.write(out + "\n")
        raise RuntimeError("command failed: " + " ".join(cmd))
    return out


def build_libjpi(verbose: bool = False) -> str:
    bdir = os.path.join(ROOT, "_build")
    os.makedirs(bdir, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
        out = _run([HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        if verbose and out.strip():
            print(out)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


def build_all(verbose: bool = False):
    sys.path.insert(0, ROOT)
    import synth
    synth.build_lib(force=True)
    lib = build_libjpi(verbose)
    # the two standalone microbenchmarks (link chains, L2 / HBM read rates)
    from paper_2607_12659_amd import l2bench, linkbench
    linkbench.build()
    l2bench.build()
    return lib


if __name__ == "__main__":
    print(build_all(verbose=True))
