"""Build libswan.so (the HIP kernels and the C ABI) for gfx950 with hipcc, and
libswanbench.so (the streaming-read ceiling that bench.py measures beside it).

Usage: python -m paper_2511_18936_amd.build   (or build() from Python)
The library is written next to this file, in-tree.
"""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libswan.so")
# measurement support (the streaming-read ceiling), a library of its own
BENCH_LIB = os.path.join(HERE, "libswanbench.so")
BENCH_SOURCES = ["stream_ceiling.hip"]
SOURCES = ["swan_api.hip", "decode.hip", "decode_gqa.hip", "decode_asym.hip",
           "decode_gqa_asym.hip", "decode_fused.hip", "compress.hip", "prefill.hip",
           "change_k.hip", "rope.hip", "calibrate.hip"]
ARCH = "gfx950"
# per-source flags: the GQA kernels and the prefill rotation keep their MFMA
# accumulators in VGPRs (the default puts them in AGPRs and copies them across
# for the VALU work on them: the per-page rescale, the per-element conversion)
SOURCE_FLAGS = {
    "decode_gqa.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "decode_gqa_asym.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
    "prefill.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
}
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    # no packed-FP32 instructions in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose: bool) -> None:
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with status {r.returncode}")


def build(verbose: bool = False, extra=()) -> str:
    """Compile every source to an object in parallel (the translation units share
    no device code), then link libswan.so; the library is replaced only on success."""
    from concurrent.futures import ThreadPoolExecutor

    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    flags = [f for f in FLAGS if f != "-shared"]
    jobs = []
    for src in SOURCES:
        obj = os.path.join(objdir, os.path.splitext(src)[0] + ".o")
        jobs.append(([hipcc(), *flags, *SOURCE_FLAGS.get(src, []), *extra, f"-I{INCLUDE}",
                      f"-I{CSRC}", "-c",
                      os.path.join(CSRC, src), "-o", obj], obj))
    workers = max(1, min(len(jobs), os.cpu_count() or 1, 8))
    with ThreadPoolExecutor(max_workers=workers) as pool:
        for f in [pool.submit(_run, cmd, verbose) for cmd, _ in jobs]:
            f.result()
    tmp = LIB + ".tmp"
    _run([hipcc(), *FLAGS, *extra, *[obj for _, obj in jobs], "-o", tmp,
          "-Wl,-rpath,/opt/rocm/lib"], verbose)
    os.replace(tmp, LIB)
    tmp = BENCH_LIB + ".tmp"
    _run([hipcc(), *FLAGS, *extra, f"-I{INCLUDE}", *[os.path.join(CSRC, s) for s in BENCH_SOURCES],
          "-o", tmp, "-Wl,-rpath,/opt/rocm/lib"], verbose)
    os.replace(tmp, BENCH_LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
