"""Compile the HIP library libmfsdp.so in-tree for gfx950 with hipcc.

Every call recompiles (no up-to-date check). The library embeds a build identifier, a SHA-256 over
its source files, the public header and the compiler flags (``mfsdp_build_id()``); the binding
refuses a library whose identifier differs from the one of the sources next to it, so a stale
binary is never run after a source change. Usage: ``python -m paper_2607_05895_amd.build_lib``.
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
LIB = os.path.join(PKG, "libmfsdp.so")
SOURCES = ["mfsdp_host.cpp", "planner.cpp", "shampoo_host.cpp", "soap_host.cpp", "kernels_elementwise.hip",
           "kernels_gemm.hip", "kernels_shampoo.hip", "kernels_soap.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed-fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


HEADER = os.path.join(ROOT, "include", "mfsdp.h")


def source_id() -> str:
    """Build identifier of the sources in the tree: SHA-256 (first 16 hex digits) over every file of
    csrc/ (sorted by name), the public header and the compiler flags. Reads files only."""
    h = hashlib.sha256()
    files = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp", ".h")))
    for name in files:
        h.update(name.encode() + b"\0")
        with open(os.path.join(CSRC, name), "rb") as f:
            h.update(f.read())
    with open(HEADER, "rb") as f:
        h.update(b"mfsdp.h\0" + f.read())
    h.update(" ".join(HIPCC_FLAGS).encode())
    return h.hexdigest()[:16]


def build(verbose: bool = False) -> str:
    """Compile every source to an object in a temporary folder (in parallel), then link them."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmpdir = tempfile.mkdtemp(prefix="mfsdp_build_")
    try:
        common = [hipcc, *HIPCC_FLAGS, f'-DMFSDP_BUILD_ID="{source_id()}"', "-I", os.path.join(ROOT, "include"),
                  "-I", CSRC]
        jobs, objs = [], []
        for src in SOURCES:
            obj = os.path.join(tmpdir, src + ".o")
            cmd = [*common, "-c", "-x", "hip", os.path.join(CSRC, src), "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            jobs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
            objs.append(obj)
        failed = []
        for src, pr in jobs:
            out, _ = pr.communicate()
            if pr.returncode != 0:
                sys.stderr.write(out)
                failed.append(src)
        if failed:
            raise RuntimeError(f"hipcc failed on {', '.join(failed)}")
        tmp = LIB + ".tmp"
        cmd = [hipcc, *HIPCC_FLAGS, *objs, "-o", tmp]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc link failed with exit code {res.returncode}")
        os.replace(tmp, LIB)
    finally:
        shutil.rmtree(tmpdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
