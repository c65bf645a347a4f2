"""Build the native parts of the package in-tree.

  libdyplan.so      the HIP library (kernels for gfx950 + C-ABI host code)
  libdyworkload.so  the seeded candidate-row generator (plain C, OpenMP)

hipcc flags: -O3 for gfx950, no fused multiply-add contraction (the fp64
re-evaluation must round exactly like the definition, operation by operation),
and packed-fp32 instruction selection disabled.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

LIB = os.path.join(HERE, "libdyplan.so")
WORKLOAD_LIB = os.path.join(HERE, "libdyworkload.so")

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
]


def _run(cmd):
    print("[build]", " ".join(cmd), flush=True)
    subprocess.check_call(cmd, cwd=ROOT)


def build_hip(extra_flags=(), out: str = LIB) -> str:
    objs = []
    for src in ("kernels.hip", "host.cpp", "jit_rows.cpp", "bundle.cpp"):
        obj = os.path.join(CSRC, "_" + src.replace(".", "_") + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        _run([HIPCC, *HIP_FLAGS, *extra_flags, f"-I{INCLUDE}", f"-I{CSRC}", *lang, "-c",
              os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", out, "-lhiprtc"])
    for o in objs:
        os.remove(o)
    return out


def build_workload() -> str:
    _run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", WORKLOAD_LIB,
          os.path.join(CSRC, "workload_rows.c")])
    return WORKLOAD_LIB


def build_all() -> None:
    build_workload()
    build_hip()


if __name__ == "__main__":
    build_all()
    sys.exit(0)
