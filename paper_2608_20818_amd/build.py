"""Build libprm.so (gfx950) in-tree with hipcc.

Each HIP source is compiled to an object in ``_build/`` in parallel, then the
objects are linked into ``libprm.so`` next to this file.  Packed fp32 VALU
instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libprm.so")
SOURCES = ("prm_api.hip", "rowwise.hip", "ns5.hip", "probe.hip", "adamw.hip")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    procs = []
    objs = []
    for s in SOURCES:
        obj = os.path.join(BUILD, s.replace(".hip", ".o"))
        objs.append(obj)
        cmd = [cc, *FLAGS, "-c", os.path.join(CSRC, s), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((s, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
    failed = []
    for s, p in procs:
        out, _ = p.communicate()
        noise = "is not a recognized feature for this target"
        lines = [ln for ln in (out or "").splitlines() if noise not in ln]
        if p.returncode != 0:
            failed.append(s)
            print("\n".join(lines), file=sys.stderr)
        elif verbose and lines:
            print("\n".join(lines))
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    tmp = LIB + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        print(r.stdout, r.stderr, file=sys.stderr)
        raise RuntimeError("link failed")
    os.replace(tmp, LIB)
    return LIB


C_CALLER_SRC = os.path.join(ROOT, "tests", "c_caller.c")
C_CALLER_LIB = os.path.join(ROOT, "tests", "libc_caller.so")


def build_c_caller() -> str:
    """The plain-C caller of the C ABI used by the GPU tests (gcc, no device
    code): tests/c_caller.c -> tests/libc_caller.so, linked to libprm.so and the
    HIP runtime."""
    cc = shutil.which("gcc") or "gcc"
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    tmp = C_CALLER_LIB + ".tmp"
    cmd = [cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-shared", "-fPIC", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "include"), "-I", os.path.join(rocm, "include"),
           C_CALLER_SRC, "-o", tmp, "-L", HERE, "-lprm", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
           f"-Wl,-rpath,$ORIGIN/../{os.path.basename(HERE)}", f"-Wl,-rpath,{os.path.join(rocm, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        print(r.stdout, r.stderr, file=sys.stderr)
        raise RuntimeError("gcc failed for tests/c_caller.c")
    os.replace(tmp, C_CALLER_LIB)
    return C_CALLER_LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
    print(build_c_caller())
