"""Build the gfx950 shared library ``libadpsgd.so`` in-tree with hipcc.

Usage: ``python -m paper_2007_06134_amd.build`` (or ``build()`` from Python).
"""
from __future__ import annotations

import hashlib
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libadpsgd.so")
ARCH = "gfx950"
ROCM_LIB = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "lib")   # roctx markers

DIGEST = LIB + ".digest"   # source digest of the library next to it

HIP_SOURCES = ["kernels.hip", "noalloc.hip"]
HOST_SOURCES = ["runtime.cpp", "controller.cpp"]


def source_digest() -> str:
    """sha256 over every file the library is built from: the sources under
    csrc/, the headers under include/ and this build script (its flags)."""
    h = hashlib.sha256()
    files = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC))]
    files += [os.path.join(INCLUDE, f) for f in sorted(os.listdir(INCLUDE))]
    files.append(os.path.abspath(__file__))
    for path in files:
        if not os.path.isfile(path):
            continue
        h.update(os.path.relpath(path, ROOT).encode() + b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()


def built_digest() -> str:
    """The source digest recorded when the library was last built ('' if none)."""
    try:
        with open(DIGEST) as f:
            return f.read().strip()
    except OSError:
        return ""


def is_current() -> bool:
    return os.path.exists(LIB) and built_digest() == source_digest()

# Packed fp32 instructions are kept out of the device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-Wall", "-Wextra", "-I", INCLUDE, "-I", CSRC]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def build(verbose: bool = False) -> str:
    cc = hipcc()
    digest = source_digest()
    with tempfile.TemporaryDirectory(prefix="adpsgd_build_") as tmp:
        objs = []
        for src in HIP_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            cmd = [cc, *COMMON, f"--offload-arch={ARCH}", "-ffp-contract=off", *DEVICE_FLAGS,
                   "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
            _run(cmd, verbose)
            objs.append(obj)
        for src in HOST_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            # the host controller takes the same fp64 decisions as the device: no contraction
            cmd = [cc, *COMMON, "-D__HIP_PLATFORM_AMD__", "-ffp-contract=off", "-c", os.path.join(CSRC, src), "-o", obj]
            _run(cmd, verbose)
            objs.append(obj)
        out_tmp = LIB + f".tmp{os.getpid()}"
        _run([cc, "-shared", f"--offload-arch={ARCH}", *objs, "-L", ROCM_LIB, "-lrocprofiler-sdk-roctx",
              f"-Wl,-rpath,{ROCM_LIB}", "-o", out_tmp], verbose)
        os.replace(out_tmp, LIB)
    tmp_digest = DIGEST + f".tmp{os.getpid()}"
    with open(tmp_digest, "w") as f:
        f.write(digest + "\n")
    os.replace(tmp_digest, DIGEST)
    return LIB


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"build step failed: {' '.join(cmd[:3])} ... {cmd[-3]}")
    if verbose and (r.stdout or r.stderr):
        sys.stderr.write(r.stdout + r.stderr)


if __name__ == "__main__":
    print(build(verbose=True))
