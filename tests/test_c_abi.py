"""A plain C program calls libswan through include/swan.h (tests/c/swan_c_example.c).

* host: size queries and argument checks from C (no GPU needed);
* gpu: compress + decode through the C ABI, checked inside the program against a
  float64 reference of Algorithm 1 computed in C (signed-permutation rotations, so
  the rotated fp32 values are exact and pruning is compared on exact values), to
  the 2e-3 bound.

The program is compiled with gcc by tests/c/build_example.py, which the package
build entry point runs after libswan.so; the host test compiles it itself if it
is missing (a CPU-only gcc step), the GPU test requires it prebuilt.
"""
import importlib.util
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c", "swan_c_example")


def _builder():
    spec = importlib.util.spec_from_file_location("swan_c_build",
                                                  os.path.join(HERE, "c", "build_example.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _run(mode):
    r = subprocess.run([EXE, mode], capture_output=True, text=True, timeout=100)
    print(r.stdout + r.stderr, flush=True)
    return r


def test_c_program_host_checks():
    src = os.path.join(HERE, "c", "swan_c_example.c")
    if not os.path.exists(EXE) or os.path.getmtime(EXE) < os.path.getmtime(src):
        _builder().build()
    r = _run("sizes")
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout + r.stderr


@pytest.mark.gpu
def test_c_program_compress_and_decode(gpu_device):
    assert os.path.exists(EXE), "tests/c/swan_c_example is not built (run the build entry point)"
    r = _run("run")
    assert r.returncode == 0 and "max relative error" in r.stdout, r.stdout + r.stderr
