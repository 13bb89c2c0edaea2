"""Build the SparsePR HIP library (libsparsepr.so) for gfx950 with hipcc.

The objects go to paper_2608_18484_amd/_build/ and the shared library next to
this file, so it travels with the source tree.
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsparsepr.so")
SOURCES = ["plan_kernels.hip", "attn_kernels.hip", "fit_kernels.hip", "noalloc.hip", "api.cpp"]
ARCH = os.environ.get("SPARSEPR_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# Packed fp32 VALU instructions are kept out of the generated code.
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-function",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str) -> subprocess.Popen:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd = [HIPCC, *FLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    return subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    procs = [(s, _compile(s)) for s in SOURCES]
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        lines = [l for l in out.splitlines() if "packed-fp32-ops" not in l]
        if p.returncode != 0:
            failed.append(src)
            sys.stderr.write("\n".join(lines) + "\n")
        elif verbose and lines:
            sys.stderr.write("\n".join(lines) + "\n")
    if failed:
        raise RuntimeError(f"hipcc failed for {failed}")
    objs = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    tmp = LIB + ".tmp"
    subprocess.check_call([HIPCC, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    return LIB


# Host-side sanitizer build: api.cpp (argument validation, workspace layout,
# export/import, timing) holds no device code, so g++ compiles it with
# AddressSanitizer and UndefinedBehaviorSanitizer and it is linked with the
# regular kernel objects into libsparsepr_san.so.  The binding loads it when
# SPARSEPR_LIB points there; the process must preload the gcc runtimes.
SAN_LIB = os.path.join(HERE, "libsparsepr_san.so")
HOST_SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=undefined"]


def build_sanitized() -> str:
    build()
    api = os.path.join(BUILD, "api_san.o")
    host_cc = ["g++", "-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]
    subprocess.check_call([*host_cc, *HOST_SAN_FLAGS, "-c", os.path.join(CSRC, "api.cpp"), "-o", api])
    objs = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "api.cpp"]
    link = ["g++", "-shared", *HOST_SAN_FLAGS, "-o", SAN_LIB, api, *objs,
            "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"]
    subprocess.check_call(link)
    return SAN_LIB


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--sanitize":
        print(build_sanitized())
    else:
        print(build(verbose=True))
