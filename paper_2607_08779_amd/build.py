"""Build libssq.so (HIP kernels + C ABI) in-tree for gfx950 with hipcc.

Usage: python -m paper_2607_08779_amd.build   (or build() from Python).
The library lands next to this file; object files go to ``_build/``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libssq.so")
# measurement-only kernels for bench.py (a streaming-read ceiling), not part of libssq
BENCH_SRC = os.path.join(PKG, "csrc_bench")
BENCH_LIB = os.path.join(PKG, "libssq_bench.so")

ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++20", "-fPIC",
    "-ffp-contract=off",                      # every fma in the kernels is written out
    # the first kernel arguments arrive in SGPRs at dispatch (no scalar load before the
    # first address is known; ~0.2 us per decode GEMV launch)
    "-mllvm", "-amdgpu-kernarg-preload-count=16",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", f"-I{INCLUDE}", f"-I{CSRC}",
]
# MFMA accumulators in VGPRs (no AGPR copies in loops); a kernel that needs AGPR
# accumulators would take an entry in FILE_FLAGS without it.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
FILE_FLAGS: dict[str, list[str]] = {}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; set HIPCC")


def sources() -> list[str]:
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _compile(src: str, build_dir: str) -> str:
    obj = os.path.join(build_dir, os.path.basename(src) + ".o")
    cmd = [hipcc(), *FLAGS, *FILE_FLAGS.get(os.path.basename(src), VGPR_FORM), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False, lib_path: str = LIB, build_dir: str = BUILD) -> str:
    """Compile every HIP source and link libssq.so (or lib_path); returns the library path.
    The default build also links bench.py's measurement library (libssq_bench.so)."""
    path = _link(sources(), lib_path, build_dir)
    if verbose:
        print(f"built {path}")
    if lib_path == LIB:
        bench_srcs = sorted(os.path.join(BENCH_SRC, f) for f in os.listdir(BENCH_SRC) if f.endswith(".hip"))
        bpath = _link(bench_srcs, BENCH_LIB, os.path.join(build_dir, "bench"))
        if verbose:
            print(f"built {bpath}")
    return path


def _link(srcs: list[str], lib_path: str, build_dir: str) -> str:
    os.makedirs(build_dir, exist_ok=True)
    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda f: _compile(f, build_dir), srcs))
    tmp = lib_path + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    # A kernel whose host launch stub the compiler did not emit links fine but fails at
    # load time; refuse such a library here.
    nm = shutil.which("nm") or "/opt/rocm/llvm/bin/llvm-nm"
    r = subprocess.run([nm, "-D", "--undefined-only", tmp], capture_output=True, text=True)
    stubs = [l for l in r.stdout.splitlines() if "__device_stub__" in l]
    if stubs:
        os.remove(tmp)
        raise RuntimeError(f"{lib_path}: kernel launch stubs missing from the host objects:\n" + "\n".join(stubs[:5]))
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
