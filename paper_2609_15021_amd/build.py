"""Build the kvx HIP library (and the harness library) for gfx950 with hipcc, in-tree.

``build_all()`` compiles every time it is called.  The CPU oracle is built by
``oracle.build()`` with gcc and is not part of this library.
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
HARNESS = os.path.join(ROOT, "harness")
BUILD_DIR = os.path.join(ROOT, "_build")

LIB_KVX = os.path.join(PKG, "libkvx.so")
LIB_HARNESS = os.path.join(HARNESS, "libkvx_harness.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed-FP32 instructions stay off in all HIP code of this project.
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wextra",
          "-Wno-unused-parameter", *NO_PACKED_FP32]

KVX_SOURCES = ["kvx_check.cpp", "kvx_engine.cpp", "kvx_gather.hip", "kvx_state.hip", "kvx_index.cpp", "kvx_tier.cpp",
               "kvx_noalloc.hip"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd)}")
    # hipcc's host pass does not know the packed-fp32 feature name; that warning is harmless.
    noise = [ln for ln in (r.stdout + r.stderr).splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "not a recognized feature" not in ln]
    if verbose and noise:
        print("\n".join(noise), flush=True)


def _compile_objs(sources, src_dir, tag, extra, verbose):
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs = []
    for src in sources:
        obj = os.path.join(BUILD_DIR, f"{tag}_{os.path.splitext(src)[0]}.o")
        _run([HIPCC, *COMMON, *extra, "-x", "hip", "-c", os.path.join(src_dir, src), "-o", obj], verbose)
        objs.append(obj)
    return objs


def _link(objs, out, verbose):
    tmp = out + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
    os.replace(tmp, out)


def build_kvx(verbose: bool = False) -> str:
    objs = _compile_objs(KVX_SOURCES, CSRC, "kvx", ["-I", INCLUDE, "-I", CSRC, "-fvisibility=hidden"], verbose)
    _link(objs, LIB_KVX, verbose)
    return LIB_KVX


def build_harness(verbose: bool = False) -> str:
    objs = _compile_objs(["harness.hip"], HARNESS, "harness", [], verbose)
    _link(objs, LIB_HARNESS, verbose)
    return LIB_HARNESS


NATIVE_SRC = os.path.join(ROOT, "tests", "native", "kvx_native_caller.c")
NATIVE_BIN = os.path.join(ROOT, "tests", "native", "kvx_native_caller")


def build_native_caller(verbose: bool = False) -> str:
    """The tests' native C caller of the C ABI (plain C against kvx.h and the HIP C API)."""
    tmp = NATIVE_BIN + ".tmp"
    _run(["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE,
          "-I", "/opt/rocm/include", NATIVE_SRC, "-o", tmp, "-L", PKG, "-lkvx",
          "-Wl,-rpath,$ORIGIN/../../paper_2609_15021_amd", "-L", "/opt/rocm/lib", "-Wl,-rpath,/opt/rocm/lib",
          "-lamdhip64"], verbose)
    os.replace(tmp, NATIVE_BIN)
    return NATIVE_BIN


TIERD_SRC = os.path.join(CSRC, "kvx_tierd.cpp")
TIERD_BIN = os.path.join(PKG, "kvx_tierd")


def build_tierd(verbose: bool = False) -> str:
    """The standalone tier daemon: a host program over the C ABI (no kernels of its own)."""
    tmp = TIERD_BIN + ".tmp"
    # libkvx.so and the HIP runtime are loaded at run time (dlopen), in that order reversed: the
    # runtime named on the command line first, so that the library binds to it.
    _run(["g++", "-std=c++17", "-O2", "-Wall", "-Wextra", "-Werror", "-I", INCLUDE, TIERD_SRC, "-o", tmp,
          "-Wl,-rpath,/opt/rocm/lib", "-ldl"], verbose)
    os.replace(tmp, TIERD_BIN)
    return TIERD_BIN


def build_all(verbose: bool = False):
    return build_kvx(verbose), build_harness(verbose), build_native_caller(verbose), build_tierd(verbose)


if __name__ == "__main__":
    print(build_all(verbose=True))
