"""Build libhils.so (gfx950) in-tree with hipcc.

    python -m paper_2607_02980_amd.build               # libhils.so
    python -m paper_2607_02980_amd.build --sanitize    # libhils_san.so (ASan/UBSan host layer)

Each source compiles to an object in ``_build/`` (in parallel), then one
shared library ``paper_2607_02980_amd/libhils.so`` is linked.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libhils.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

SOURCES = ["hils_api.cpp", "hils_fwd.hip", "hils_prefill.hip", "hils_bwd.hip", "hils_bwd_mfma.hip", "hils_decode.hip", "hils_landmark.hip", "hils_noalloc.hip"]

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 ALU ops are kept out of the generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", os.path.join(ROOT, "include"),
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"] if src.endswith(".hip") else []
    cmd = [HIPCC, *FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed on {src}")
    if verbose and r.stderr.strip():
        sys.stderr.write(r.stderr)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = [s for s in SOURCES if os.path.exists(os.path.join(CSRC, s))]
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


SAN_LIB = os.path.join(PKG, "libhils_san.so")


def build_sanitized(verbose: bool = False) -> str:
    """libhils_san.so: the host layer (hils_api.cpp: argument checks, workspace
    sizing, dispatch) compiled under AddressSanitizer and UndefinedBehaviorSanitizer
    (host code only), linked with the regular kernel objects.  Loaded through
    HILS_LIB by a process that preloads clang's ASan runtime."""
    objs = [os.path.join(BUILD, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    if not all(os.path.exists(o) for o in objs):
        build(verbose)
    san_dir = os.path.join(BUILD, "san")
    os.makedirs(san_dir, exist_ok=True)
    api_obj = os.path.join(san_dir, "hils_api.o")
    cmd = [HIPCC, *FLAGS, "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-c", os.path.join(CSRC, "hils_api.cpp"), "-o", api_obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed on the sanitized hils_api.cpp")
    objs = [api_obj if o.endswith("hils_api.o") else o for o in objs]
    tmp = SAN_LIB + ".tmp"
    subprocess.check_call([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_sanitized(verbose="-v" in sys.argv))
    else:
        print(build(verbose="-v" in sys.argv))
