"""Compile swan_c_example.c, a plain C caller of libswan, with gcc.

The program includes only include/swan.h and the HIP runtime's C header and links
the in-tree libswan.so (found at run time through an $ORIGIN-relative rpath), so
it checks that the boundary is usable from C with no C++ or Python in between.
Usage: python tests/c/build_example.py   (libswan.so must be built first)
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "swan_c_example.c")
EXE = os.path.join(HERE, "swan_c_example")
PKG = os.path.join(ROOT, "paper_2511_18936_amd")


def build(verbose: bool = False) -> str:
    if not os.path.exists(os.path.join(PKG, "libswan.so")):
        raise RuntimeError("libswan.so is not built")
    rel = os.path.relpath(PKG, HERE)
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROOT, 'include')}", "-I/opt/rocm/include", SRC, "-o", EXE + ".tmp",
           f"-L{PKG}", "-lswan", "-L/opt/rocm/lib", "-lamdhip64", "-lm",
           f"-Wl,-rpath,$ORIGIN/{rel}", "-Wl,-rpath,/opt/rocm/lib"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"gcc failed with status {r.returncode}")
    os.replace(EXE + ".tmp", EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
