"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two builds, made here with the host compilers, sanitizers on host code only
(nothing here is device code):

* the oracle (oracle/swr_oracle.c), which indexes [T][D] arrays by hand,
  driven by the oracle's pin tests;
* the C ABI's validation and launch planning (swr_api.cpp: 64-bit size,
  stride, overlap and alias arithmetic on caller-provided values), linked
  with host stand-ins for the kernel launchers (sanitize/launch_stub.cpp)
  and driven by the ABI tests plus a sweep of valid calls through every
  entry point (sanitize/sweep_valid.py).

Each suite runs in a child process with the sanitizer runtime preloaded and
the sanitized library swapped in for the normal one; any report aborts the
child, which fails the test.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _runtime(name):
    gcc = shutil.which("gcc")
    if not gcc:
        return None
    path = subprocess.run([gcc, f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


LIBASAN = _runtime("libasan.so")
pytestmark = pytest.mark.skipif(LIBASAN is None or shutil.which("g++") is None,
                                reason="gcc's sanitizer runtimes are not installed")

# Child: swap the sanitized builds in before anything loads a library, then run pytest.
RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle, oracle.build
import paper_2512_13921_amd as swr, paper_2512_13921_amd.build
if {oracle_lib!r}:
    oracle.build.LIB = {oracle_lib!r}
if {api_lib!r}:
    paper_2512_13921_amd.build.LIB = {api_lib!r}
import pytest
rc = pytest.main(["-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu", "--rootdir", {root!r}] + {tests_list!r})
# which of the libraries the tests actually ran on
for line in open("/proc/self/maps"):
    if "libswr" in line:
        print("MAPPED", line.split()[-1])
sys.exit(rc)
"""


def _child(tmp_path, tests, oracle_lib="", api_lib=""):
    code = RUNNER.format(root=ROOT, tests=HERE, oracle_lib=oracle_lib, api_lib=api_lib,
                         tests_list=[os.path.join(HERE, t) for t in tests])
    env = dict(os.environ)
    env["LD_PRELOAD"] = LIBASAN
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "4"
    res = subprocess.run([sys.executable, "-c", code], cwd=str(tmp_path), env=env, capture_output=True,
                         text=True, timeout=900)
    out = res.stdout + res.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert res.returncode == 0, out[-6000:]
    return out


def test_oracle_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "libswr_oracle_san.so")
    subprocess.run(["gcc", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", *SAN,
                    os.path.join(ROOT, "oracle", "swr_oracle.c"), "-o", lib], check=True)
    out = _child(tmp_path, ["test_oracle.py", "test_oracle_exact.py", "test_oracle_step.py",
                            "test_oracle_uniform.py", "test_oracle_groups.py"], oracle_lib=lib)
    assert " passed" in out and f"MAPPED {lib}" in out, out[-3000:]
    assert "MAPPED " + os.path.join(ROOT, "oracle", "libswr_oracle.so") not in out


def test_abi_validation_under_asan_ubsan(tmp_path):
    lib = str(tmp_path / "libswr_hostcheck.so")
    csrc = os.path.join(ROOT, "paper_2512_13921_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-fPIC", "-shared", *SAN, "-D__HIP_PLATFORM_AMD__",
                    "-I/opt/rocm/include", os.path.join(csrc, "swr_api.cpp"),
                    os.path.join(HERE, "sanitize", "launch_stub.cpp"), "-o", lib], check=True)
    out = _child(tmp_path, ["test_abi.py", os.path.join("sanitize", "sweep_valid.py")], api_lib=lib)
    assert " passed" in out and f"MAPPED {lib}" in out, out[-3000:]
    assert "MAPPED " + os.path.join(ROOT, "paper_2512_13921_amd", "libswr.so") not in out
