"""Build libadapld.so for gfx950 with hipcc (in-tree, next to this file).

    python -m paper_2606_05742_amd.build

Every call recompiles every source.  Objects go to ``_build/`` beside the
sources; the shared library lands in this package directory.
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
LIB = os.path.join(PKG, "libadapld.so")

SOURCES = ["lexical.hip", "semantic.hip", "tree.hip", "paper_tree.hip", "verify.hip", "accept.hip", "embed.hip", "ngram.hip", "noalloc.hip", "abi.cpp"]
ARCH = "gfx950"

# -packed-fp32-ops keeps the compiler from emitting packed fp32 VALU ops.
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP toolchain is required to build libadapld")


# Inputs of the verify attention are finite by contract, so its max reductions
# need no NaN canonicalisation (v_max3 chains without quieting operations).
PER_SOURCE_FLAGS = {"verify.hip": ["-fno-honor-nans"]}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    extra = PER_SOURCE_FLAGS.get(src, [])
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(min(len(SOURCES), 8)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


# The host-side C-ABI glue built with AddressSanitizer and UBSan (gcc, host
# code only) and linked with the regular objects: a test library for the
# argument-validation paths, loaded with the gcc sanitizer runtimes preloaded.
HOSTSAN_LIB = os.path.join(BUILD, "libadapld_hostsan.so")
HOSTSAN_FLAGS = ["-O1", "-g", "-std=c++17", "-fPIC", "-fno-omit-frame-pointer", "-fsanitize=address,undefined"]


def build_host_sanitized() -> str:
    """libadapld with abi.cpp compiled by g++ under ASan + UBSan; the kernels'
    objects are the regular ones (built first when missing)."""
    objs = [os.path.join(BUILD, os.path.splitext(src)[0] + ".o") for src in SOURCES if src != "abi.cpp"]
    if not all(os.path.exists(o) for o in objs):
        build()
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    san_obj = os.path.join(BUILD, "abi_hostsan.o")
    cmd = ["g++", *HOSTSAN_FLAGS, "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(rocm, "include"), "-I", INCLUDE,
           "-I", CSRC, "-x", "c++", "-c", os.path.join(CSRC, "abi.cpp"), "-o", san_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized compile of abi.cpp failed:\n{r.stderr}")
    cmd = ["g++", "-shared", "-fsanitize=address,undefined", "-o", HOSTSAN_LIB, san_obj, *objs,
           "-L", os.path.join(rocm, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(rocm, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{r.stderr}")
    return HOSTSAN_LIB


def sanitizer_preload() -> str:
    """LD_PRELOAD value for a process that loads HOSTSAN_LIB."""
    libs = []
    for name in ("libasan.so", "libubsan.so"):
        out = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
        libs.append(out)
    return ":".join(libs)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
