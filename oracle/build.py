"""Build the double-precision CPU oracle (test infrastructure) into
``oracle/libswr_oracle.so`` with the host C compiler and OpenMP.

Usage: ``python oracle/build.py``.  Building the checker is not using it; the
package build step calls this too so that the checker exists on every machine
the tests run on.
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "swr_oracle.c")
LIB = os.path.join(HERE, "libswr_oracle.so")


def build(verbose: bool = False) -> str:
    cc = os.environ.get("CC", "gcc")
    # -ffp-contract=off keeps every product and sum a separately rounded double
    # operation, exactly as written in the source.
    cmd = [cc, "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-Wall", "-Wextra", SRC, "-o", LIB + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(LIB + ".tmp", LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    lib_t = os.path.getmtime(LIB)
    return any(os.path.getmtime(os.path.join(HERE, f)) > lib_t
               for f in ("swr_oracle.c", "swr_oracle.h"))


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
