"""Build step of the HIP libraries: hipcc for gfx950, in-tree.

    python -m paper_2609_34117_amd.build

compiles every ``csrc/*.hip`` to an object under ``_build/`` (in parallel)
and links ``paper_2609_34117_amd/libslimwise.so`` (the MoE layer), and
``gen/*.hip`` into ``paper_2609_34117_amd/libswgen.so`` (device draws of
synthetic inputs, kept apart from the layer).
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD_DIR = os.path.join(ROOT, "_build", "slimwise")
LIB = os.path.join(PKG, "libslimwise.so")
GEN_SRC = os.path.join(PKG, "gen")
GEN_BUILD_DIR = os.path.join(ROOT, "_build", "swgen")
GEN_LIB = os.path.join(PKG, "libswgen.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# gfx950 only.  Packed-fp32 VALU forms are disabled: hipcc would otherwise
# generate v_pk_{add,mul,fma}_f32 from plain float code.
HIP_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I" + os.path.join(ROOT, "include"),
]


def sources(src_dir: str = CSRC) -> list[str]:
    return sorted(os.path.join(src_dir, f) for f in os.listdir(src_dir) if f.endswith(".hip"))


def _compile(src: str, build_dir: str) -> str:
    obj = os.path.join(build_dir, os.path.basename(src)[:-4] + ".o")
    cmd = [HIPCC, *HIP_FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def _build_lib(src_dir: str, build_dir: str, lib: str) -> str:
    os.makedirs(build_dir, exist_ok=True)
    srcs = sources(src_dir)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, build_dir), srcs))
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    return lib


def build(verbose: bool = False) -> str:
    """Compile and link libslimwise.so and libswgen.so; returns the former's path."""
    _build_lib(CSRC, BUILD_DIR, LIB)
    _build_lib(GEN_SRC, GEN_BUILD_DIR, GEN_LIB)
    if verbose:
        print(f"built {LIB} and {GEN_LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
