"""Host code under AddressSanitizer and UBSan (no GPU): the fp64 oracle
(oracle.c, objective.c) and the library's host-only code (validation, dry
staging and the kernel-source generator, suffix recompilation, bundle
annotations, the switching simulator, self checks) are built with the
sanitizers into two small drivers (tests/sanitize/) that call every entry
point on seeded problems; both must exit 0 with no sanitizer report."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_02942_amd", "csrc")
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def run(exe):
    res = subprocess.run([exe], capture_output=True, text=True, env=ENV, timeout=300)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    for marker in ("runtime error", "AddressSanitizer", "LeakSanitizer"):
        assert marker not in res.stderr, res.stderr[-4000:]
    return res.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not installed")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.check_call(["gcc", "-std=c11", "-ffp-contract=off", *SAN,
                           os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"), "-o", exe, "-lm"])
    assert "0 failed calls" in run(exe)


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime.h"), reason="HIP headers not installed")
def test_library_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_driver")
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                           f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
                           os.path.join(CSRC, "host.cpp"), os.path.join(CSRC, "jit_rows.cpp"),
                           os.path.join(CSRC, "bundle.cpp"), os.path.join(ROOT, "tests", "sanitize", "host_driver.cpp"),
                           "-o", exe, "-L/opt/rocm/lib", "-lamdhip64", "-lhiprtc", "-Wl,-rpath,/opt/rocm/lib"])
    assert "0 failed checks" in run(exe)
