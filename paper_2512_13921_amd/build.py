"""Build the gfx950 HIP library ``paper_2512_13921_amd/libswr.so``.

Usage: ``python -m paper_2512_13921_amd.build`` (or ``python paper_2512_13921_amd/build.py``).
Cross-compiles on a machine without a GPU.
"""
import os
import re
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libswr.so")
SOURCES = [os.path.join(CSRC, n) for n in ("swr_api.cpp", "swr_kernels.hip", "swr_uniform.hip", "swr_groups.hip",
                                            "swr_noalloc.hip", "swr_chain.hip")]
HEADERS = [os.path.join(CSRC, "swr_launch.h"), os.path.join(CSRC, "swr_device.h"),
           os.path.join(CSRC, "swr_internal.h"),
           os.path.join(os.path.dirname(HERE), "include", "swr.h")]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (set HIPCC or install ROCm)")


FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
         # no packed-fp32 instructions in device code (host pass ignores the feature)
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function"]


# Kernels that must compile without register spills: the forward sweeps copy
# their next tiles straight into LDS, and a forward instantiation that spilled
# was once measured writing wrong outputs; the one-pass exact forwards are
# held to register caps (two or three workgroups a compute unit) that a
# spill would silently turn into scratch traffic.  The build refuses any such
# spill.
NO_SPILL = ("swr_fwd_kernel", "swr_fwd_chain_kernel", "swr_fwd_chain_pair_kernel", "swr_fwd_chain_pc_kernel")
NO_SPILL_SOURCES = ("swr_kernels.hip", "swr_chain.hip")
RESOURCE_REMARKS = "-Rpass-analysis=kernel-resource-usage"


def compile_command(src: str, obj: str, extra=()) -> list:
    remarks = [RESOURCE_REMARKS] if os.path.basename(src) in NO_SPILL_SOURCES else []
    return [hipcc(), *FLAGS, *remarks, *extra, "-c", src, "-o", obj]


def spilled_kernels(text: str) -> list:
    """Mangled names of NO_SPILL kernels whose resource remarks report scratch."""
    bad, name = [], None
    for line in text.splitlines():
        if "Function Name: " in line:
            name = line.split("Function Name: ", 1)[1].split()[0]
        elif name and "ScratchSize [bytes/lane]: " in line:
            size = int(line.split("ScratchSize [bytes/lane]: ", 1)[1].split()[0])
            if size > 0 and any(k in name for k in NO_SPILL):
                bad.append(f"{name} ({size} bytes/lane)")
            name = None
    return bad


def link_command(objs, out: str) -> list:
    return [hipcc(), f"--offload-arch={ARCH}", "-shared", *objs, "-o", out]


def _messages(res) -> list:
    # hipcc's host pass warns that it does not know the packed-fp32 feature;
    # the resource remarks are read by spilled_kernels, not shown
    noise = ("is not a recognized feature for this target", "remark: ", "-Rpass-analysis")
    quoted = re.compile(r"^\s*\d*\s*\|")   # the source lines a remark quotes
    return [ln for ln in (res.stdout + res.stderr).splitlines()
            if not any(n in ln for n in noise) and not quoted.match(ln)]


def build(verbose: bool = False, extra=(), out: str = LIB) -> str:
    """Compiles every source to an object (in parallel), then links ``out``."""
    with tempfile.TemporaryDirectory() as tmp:
        objs = [os.path.join(tmp, os.path.basename(s) + ".o") for s in SOURCES]
        procs = []
        for src, obj in zip(SOURCES, objs):
            cmd = compile_command(src, obj, extra)
            if verbose:
                print(" ".join(cmd))
            procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.PIPE, text=True))
        failed = []
        for proc in procs:
            stdout, stderr = proc.communicate()
            res = subprocess.CompletedProcess(proc.args, proc.returncode, stdout, stderr)
            msgs = _messages(res)
            if res.returncode != 0:
                failed.append("\n".join(msgs))
            elif verbose and msgs:
                print("\n".join(msgs))
            spills = spilled_kernels(res.stdout + res.stderr)
            if spills:
                failed.append("kernels that must not spill registers do:\n  " + "\n  ".join(spills))
        if failed:
            raise RuntimeError("hipcc failed:\n" + "\n".join(failed))
        cmd = link_command(objs, out + ".tmp")
        if verbose:
            print(" ".join(cmd))
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("hipcc link failed:\n" + "\n".join(_messages(res)))
    os.replace(out + ".tmp", out)
    return out


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(f) > t for f in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True))
