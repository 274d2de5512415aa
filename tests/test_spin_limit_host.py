"""The one-pass exact recurrence's poll limit, as the host hands it to the
launchers (CPU only).

A chunk of the one-pass forward or backward waits for earlier chunks'
publications for at most 2^16 polls; the environment variable
SWR_CHAIN_SPIN_LIMIT may lower that (tests force the time-out path with it)
but never raise it, and a value that is not a plain integer in [0, 65535]
is ignored.  The C ABI is built here for the CPU with host stand-ins for the
launchers (sanitize/launch_stub.cpp), which check the limit they receive
against SWR_STUB_EXPECT_SPIN_LIMIT and abort on a mismatch; the calls run in
a child process, since an abort ends it.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                                reason="needs g++ and the ROCm headers")

# (SWR_CHAIN_SPIN_LIMIT, the limit the launchers must receive); None: unset
CASES = [(None, 65536), ("0", 0), ("1", 1), ("100", 100), ("65535", 65535), ("65536", 65536),
         ("1000000", 65536), ("-5", 65536), ("abc", 65536), ("12x", 65536), ("", 65536),
         (" 7", 7), ("+9", 9)]   # (leading blanks and a sign are read as strtol reads them)

CHILD = r"""
import ctypes, os, sys
sys.path[:0] = [{root!r}]
import paper_2512_13921_amd as swr, paper_2512_13921_amd.build
paper_2512_13921_amd.build.LIB = {lib!r}
lib = swr.load()
GB = 1 << 30
X, A, B_, C, Y, DY, DX, DA, DB, DC, V, WS = (ctypes.c_void_p(GB * 4 * (i + 1)) for i in range(12))
E_HIP = -8

def problem(T, H, D):
    return swr.make_problem(1, T, H, D, 128, swr.SWR_DTYPE_BF16, (T * H * D, H * D, D), (T * H, H, 1))

for value, want in {cases!r}:
    if value is None:
        os.environ.pop("SWR_CHAIN_SPIN_LIMIT", None)
    else:
        os.environ["SWR_CHAIN_SPIN_LIMIT"] = value
    os.environ["SWR_STUB_EXPECT_SPIN_LIMIT"] = str(want)
    # heads of 128 channels: the chained forward; of 64: the paired-head
    # forward and the one-pass backward
    p128, p64 = problem(4096, 2, 128), problem(4096, 2, 64)
    assert lib.swr_exact_forward(ctypes.byref(p128), X, A, B_, C, None, Y, V, None, WS, None) == E_HIP
    assert lib.swr_exact_forward(ctypes.byref(p64), X, A, B_, C, None, Y, V, None, WS, None) == E_HIP
    assert lib.swr_exact_backward(ctypes.byref(p64), X, A, B_, C, DY, None, V, None, DX, DA, DB, DC, None,
                                  WS, None) == E_HIP
    print("case", repr(value), "->", want, flush=True)
print("MAPPED", [l.split()[-1] for l in open("/proc/self/maps") if "libswr" in l][0])
"""


@pytest.fixture(scope="module")
def stub_lib(tmp_path_factory):
    lib = str(tmp_path_factory.mktemp("stub") / "libswr_hoststub.so")
    csrc = os.path.join(ROOT, "paper_2512_13921_amd", "csrc")
    subprocess.run(["g++", "-std=c++17", "-O1", "-fPIC", "-shared", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    os.path.join(csrc, "swr_api.cpp"), os.path.join(HERE, "sanitize", "launch_stub.cpp"),
                    "-o", lib], check=True)
    return lib


def _run(lib, cases, tmp_path):
    env = {k: v for k, v in os.environ.items() if k not in ("SWR_CHAIN_SPIN_LIMIT", "SWR_STUB_EXPECT_SPIN_LIMIT")}
    code = CHILD.format(root=ROOT, lib=lib, cases=cases)
    return subprocess.run([sys.executable, "-c", code], cwd=str(tmp_path), env=env, capture_output=True,
                          text=True, timeout=300)


def test_the_limit_can_only_be_lowered(stub_lib, tmp_path):
    res = _run(stub_lib, CASES, tmp_path)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert out.count("case ") == len(CASES), out[-4000:]
    assert f"MAPPED {stub_lib}" in out, out[-4000:]


def test_the_stub_check_is_live(stub_lib, tmp_path):
    # a deliberately wrong expectation must stop the child in the launcher
    res = _run(stub_lib, [("50", 51)], tmp_path)
    assert res.returncode != 0
    assert "look-back poll limit not the expected one" in res.stderr, res.stderr[-4000:]
