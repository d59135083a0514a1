"""Build libcsr.so (HIP kernels + C ABI) for gfx950 in-tree with hipcc.

``python -m paper_2605_07325_amd.build`` compiles every source under ``csrc/``
into ``paper_2605_07325_amd/libcsr.so``, and the benchmark-support sources under
``bench_csrc/`` (a measured MFMA ceiling) into ``libcsr_bench.so``.  It always
recompiles.
"""
from __future__ import annotations

import concurrent.futures
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libcsr.so")
BENCH_CSRC = os.path.join(PKG, "bench_csrc")
BENCH_LIB = os.path.join(PKG, "libcsr_bench.so")
ROOT = os.path.dirname(PKG)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed-fp32 instructions stay disabled: the compiler may not form them.
CFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def _compile(src: str, obj_dir: str = OBJ, defines=()) -> str:
    obj = os.path.join(obj_dir, os.path.basename(src) + ".o")
    cmd = [HIPCC, *CFLAGS, *[f"-D{d}" for d in defines], "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, out: str = LIB, defines=(), src_dir: str = CSRC) -> str:
    """Compile every source of ``src_dir`` and link ``out``; ``defines`` are extra -D macros."""
    obj_dir = OBJ if out == LIB else (os.path.join(OBJ, "bench") if out == BENCH_LIB else out + ".objs")
    os.makedirs(obj_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(src_dir, "*.hip")) + glob.glob(os.path.join(src_dir, "*.cpp")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, obj_dir, defines), srcs))
    tmp = out + ".tmp"
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


def build_bench(verbose: bool = False) -> str:
    """Benchmark-support library (not part of the C ABI of libcsr)."""
    return build(verbose=verbose, out=BENCH_LIB, src_dir=BENCH_CSRC)


if __name__ == "__main__":
    build(verbose=True)
    build_bench(verbose=True)
    sys.exit(0)
