"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only, no GPU needed).

Every source of the library is compiled again with both sanitizers on its
host code (device code is compiled as usual and never runs here) and linked
with tests/abi_host_check.cpp, a program that drives the C ABI through its
host-side paths: argument validation of every entry point, the workspace
size arithmetic over a sweep of shapes, status strings, the profiler's
bookkeeping and the per-thread error detail from several threads.  A
sanitizer report, a leak or a failed check fails the test.
"""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_01563_amd", "csrc")
INCLUDE = os.path.join(ROOT, "include")
CHECK_SRC = os.path.join(ROOT, "tests", "abi_host_check.cpp")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

# sanitizers on the host side of every compile and of the link only
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
       "-fno-omit-frame-pointer"]
HOST_CXX = ["-x", "c++", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include")]
DEVICE = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc():
    path = shutil.which("hipcc") or os.path.join(ROCM, "bin", "hipcc")
    if not os.path.exists(path):
        pytest.skip("hipcc not available")
    return path


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, "%s\n%s" % (" ".join(cmd), r.stderr[-4000:])


@pytest.fixture(scope="module")
def sanitized_check(tmp_path_factory):
    out = tmp_path_factory.mktemp("asan")
    hipcc = _hipcc()
    common = ["-O1", "-g", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC, *SAN]
    jobs = []
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "conv", "*.hip")))
    for src in srcs:
        obj = str(out / (os.path.basename(src) + ".o"))
        jobs.append((subprocess.Popen([hipcc, *common, *DEVICE, "-c", src, "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.PIPE), obj))
    for src in sorted(glob.glob(os.path.join(CSRC, "*.cpp")) +
                      glob.glob(os.path.join(CSRC, "conv", "*.cpp"))) + [CHECK_SRC]:
        obj = str(out / (os.path.basename(src) + ".o"))
        jobs.append((subprocess.Popen([hipcc, *common, *HOST_CXX, "-c", src, "-o", obj],
                                      stdout=subprocess.PIPE, stderr=subprocess.PIPE), obj))
    objs = []
    for proc, obj in jobs:
        _, err = proc.communicate()
        assert proc.returncode == 0, err.decode()[-4000:]
        objs.append(obj)
    exe = str(out / "abi_host_check")
    _run([hipcc, *SAN, "--offload-arch=gfx950", *objs, "-o", exe,
          "-Wl,-rpath," + os.path.join(ROCM, "lib")])
    return exe


def test_host_code_clean_under_asan_and_ubsan(sanitized_check):
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:abort_on_error=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sanitized_check], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-6000:]
    assert "abi host checks passed" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr
