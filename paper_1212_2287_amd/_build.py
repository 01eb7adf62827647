"""Build of the HIP library ``libtreeens.so`` (gfx950), in-tree next to this file."""
from __future__ import annotations

import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libtreeens.so")

# Device code: gfx950 only, IEEE single-precision denormals kept (the strict tie rule stores
# the float after 0.0, a subnormal), packed-fp32 instructions disabled.
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-fno-gpu-flush-denormals-to-zero",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; the gfx950 library cannot be built")


def build(out: str = LIB, verbose: bool = False) -> str:
    """Compile the packer and the code generator (host C++) and the kernels + C ABI (HIP) into
    one shared library (linked with hiprtc for the model-specialised kernels)."""
    tmp = out + ".tmp"
    run = (lambda c: subprocess.run(c, check=True)) if verbose else \
        (lambda c: subprocess.run(c, check=True, stdout=subprocess.DEVNULL))
    objs = []
    for name in ("pack", "codegen"):
        o = f"{out}.{name}.o"
        run(["g++", "-O2", "-std=c++17", "-fPIC", "-Wall", "-Werror", "-c",
             os.path.join(CSRC, f"{name}.cpp"), "-o", o])
        objs.append(o)
    run([_hipcc(), *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-shared",
         os.path.join(CSRC, "tree_ens.hip"), os.path.join(CSRC, "topk.hip"), "-x", "none", *objs,
         "-lhiprtc", "-o", tmp])
    os.replace(tmp, out)
    for o in objs:
        os.remove(o)
    return out


C_CLIENT_SRC = os.path.join(ROOT, "tests", "c_client.c")
C_CLIENT = os.path.join(ROOT, "tests", "c_client")


def build_c_client(out: str = C_CLIENT, lib_dir: str = PKG) -> str:
    """Compile the plain-C test client of the C ABI (gcc, no HIP device code) against the
    built library; it finds the library next to this file through its run path."""
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(_hipcc())))
    rel = os.path.relpath(lib_dir, os.path.dirname(os.path.abspath(out)))
    subprocess.run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
                    "-I", INCLUDE, "-I", os.path.join(rocm, "include"), C_CLIENT_SRC, "-o", out,
                    "-L", lib_dir, "-ltreeens", "-L", os.path.join(rocm, "lib"), "-lamdhip64",
                    f"-Wl,-rpath,$ORIGIN/{rel}", "-Wl,-rpath," + os.path.join(rocm, "lib")], check=True)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_c_client())
