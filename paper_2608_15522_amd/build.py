"""Build libsa.so (the HIP kernels and the C ABI) for gfx950 in-tree.

Usage: ``python -m paper_2608_15522_amd.build`` or ``build()`` from Python.
Every call compiles from source (one object per ``csrc/*.hip``, in parallel)
and links ``paper_2608_15522_amd/libsa.so``.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

try:
    from .srcid import source_id
except ImportError:  # run as a script
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    from paper_2608_15522_amd.srcid import source_id

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libsa.so")
BENCH_SRC = os.path.join(CSRC, "bench", "sa_bench.hip")
BENCH_LIB = os.path.join(PKG, "libsa_bench.so")

ARCH = os.environ.get("SA_OFFLOAD_ARCH", "gfx950")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 VALU instructions are kept out of the generated code.
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(src: str, defines=()) -> str:
    obj = os.path.join(OBJ, os.path.basename(src).replace(".hip", ".o"))
    cmd = [HIPCC, *CFLAGS, *defines, "-c", src, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{res.stderr}")
    return obj


def _link(objs, lib: str) -> None:
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stderr}")
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    """Builds libsa.so (the attention path) and libsa_bench.so (the MFMA
    throughput probe used by the benchmark)."""
    os.makedirs(OBJ, exist_ok=True)
    srcs = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                  if f.endswith(".hip"))
    # the library reports the sources it was built from (sa_build_id)
    defines = [f'-DSA_SRC_ID="{source_id()}"']
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs) + 1)) as ex:
        objs = list(ex.map(lambda f: _compile(f, defines), srcs + [BENCH_SRC]))
    _link(objs[:-1], LIB)
    _link(objs[-1:], BENCH_LIB)
    if verbose:
        print(f"built {LIB} and {BENCH_LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
