"""The kernels the library generates per problem (compiled at run time with
hiprtc on the device) compile offline for gfx950 with the same options, and
use no scratch memory or dynamic stack: every per-lane value stays in
registers, also around the out-of-line per-level CP function of per-backend
pressure.  Host-only: dy_kernel_source derives the problem's constants without
a device."""
import os
import re
import subprocess
import tempfile

import numpy as np
import pytest

from paper_2607_02942_amd import dyplan as D
from paper_2607_02942_amd import workload as wl

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# the options jit_rows.cpp hands to hiprtc, which also includes the HIP runtime header itself
FLAGS = ["--offload-arch=gfx950", "-O3", "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang",
         "-packed-fp32-ops", "--cuda-device-only", "-x", "hip", "-c", "-Rpass-analysis=kernel-resource-usage"]


def cases():
    out = []
    for name in ("chain4", "forkjoin8", "layered10", "stream24"):
        out.append((name, "level"))
        out.append((name, "per-class"))
        out.append((name, "objective"))
    out.append(("batch6[7]", "level"))
    return out


def problem(name, mode):
    prob = wl.batch6_request(7) if name == "batch6[7]" else wl.by_name(name)
    if mode == "per-class":
        return wl.per_class(prob)
    if mode == "objective":
        return (prob, wl.paper_objective(prob))
    return prob


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
@pytest.mark.parametrize("name,mode", cases())
def test_generated_kernels_compile_without_scratch(name, mode):
    prob = problem(name, mode)
    src = D.kernel_source(prob)
    kernels = set(re.findall(r'extern "C" __global__ void __launch_bounds__\(256\) (\w+)\(', src))
    assert {"dy_rows_scan_a", "dy_rows_scan_u", "dy_rows_sample", "dy_sweep"} <= kernels
    if mode != "per-class":
        assert "dy_score_rows" in kernels and "dy_score_range" not in kernels
    if mode == "level":
        assert "dy_sweep_seed" in kernels
    with tempfile.TemporaryDirectory() as td:
        path = os.path.join(td, "gen.hip")
        with open(path, "w") as f:
            f.write("#include <hip/hip_runtime.h>\n" + src)
        res = subprocess.run([HIPCC, *FLAGS, path, "-o", os.path.join(td, "gen.o")], capture_output=True, text=True)
    assert res.returncode == 0, res.stderr[-2000:]
    rem = res.stderr
    names = re.findall(r"remark:\s+Function Name: (\w+)", rem)
    assert kernels <= set(names), (kernels, names)
    scratch = [int(x) for x in re.findall(r"ScratchSize \[bytes/lane\]: (\d+)", rem)]
    dyn = re.findall(r"Dynamic Stack: (\w+)", rem)
    assert len(scratch) == len(names) and all(s == 0 for s in scratch), list(zip(names, scratch))
    assert all(d == "False" for d in dyn), list(zip(names, dyn))


def test_kernel_source_rejects_invalid_problems():
    prob = wl.chain4()
    prob.edges = np.array([[2, 1]], np.int32)
    with pytest.raises(D.DyplanError) as e:
        D.kernel_source(prob)
    assert e.value.args[0] == D.DY_ENOTDAG or "DY_ENOTDAG" in str(e.value) or "-2" in str(e.value)
