"""Build libcurvefp.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2608_10010_amd.build

Every call recompiles.  First the table generator (csrc/gen_tables.cpp with the
derivation in csrc/tables.cpp, host C++) is built with g++ and run: it writes the
constant tables as initializers (_build/gen/curvefp_tables.inc) and stops the
build if one of the derivation's checks fails.  The kernel sources then hold the
tables as compile-time __constant__ arrays.  The library lands in
paper_2608_10010_amd/_build/.
"""

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(BUILD, "libcurvefp.so")
SOURCES = ["api.cpp", "quantize.hip", "dequantize.hip", "gemm.hip", "scratch.hip"]
GEN_SOURCES = ["gen_tables.cpp", "tables.cpp"]
GEN_DIR = os.path.join(BUILD, "gen")
TABLES_INC = os.path.join(GEN_DIR, "curvefp_tables.inc")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    # no packed fp32 instructions anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def cxx() -> str:
    for cand in (os.environ.get("CXX"), shutil.which("g++"), "/usr/bin/g++"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("g++ not found")


def build_generator(out_dir: str, verbose: bool = False) -> str:
    """Compile the host table generator into out_dir; returns its path."""
    os.makedirs(out_dir, exist_ok=True)
    exe = os.path.join(out_dir, "gen_tables")
    cmd = [cxx(), "-O2", "-std=c++17", "-Wall", "-o", exe] + [os.path.join(CSRC, f) for f in GEN_SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return exe


def generate_tables(verbose: bool = False) -> str:
    exe = build_generator(BUILD, verbose)
    os.makedirs(GEN_DIR, exist_ok=True)
    tmp = TABLES_INC + ".tmp"
    subprocess.run([exe, tmp], check=True)
    os.replace(tmp, TABLES_INC)
    return TABLES_INC


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    generate_tables(verbose)
    cc = hipcc()

    def compile_one(src: str) -> str:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [cc] + HIPCC_FLAGS + lang + ["-I", os.path.join(ROOT, "include"), "-I", GEN_DIR, "-c",
                                           os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        return obj

    # the translation units are independent: compile them side by side
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as pool:
        objs = list(pool.map(compile_one, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
