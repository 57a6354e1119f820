"""Builds libegmla.so (the EG-MLA C-ABI library) for gfx950 with hipcc, in-tree.

    python -m paper_2509_16686_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libegmla.so")

SOURCES = ["host_plan.cpp", "decode.hip", "append.hip", "prefill.hip", "gate.hip", "literal.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # keep fp32 arithmetic out of packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


PROBE = os.path.join(PKG, "stream_probe")


def build_probe(verbose: bool = False) -> str:
    """Compiles the streaming-read reference (csrc/stream_probe.hip, not part of the library)."""
    fd, tmp = tempfile.mkstemp(dir=PKG, prefix=".stream_probe.")
    os.close(fd)
    flags = [f for f in HIPCC_FLAGS if f not in ("-fPIC", "-shared")]
    cmd = [hipcc(), *flags, os.path.join(CSRC, "stream_probe.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        os.unlink(tmp)
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with exit code {r.returncode}")
    os.chmod(tmp, 0o755)
    os.replace(tmp, PROBE)
    return PROBE


def build(verbose: bool = False) -> str:
    """Compiles every source into libegmla.so next to this file; returns its path."""
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    fd, tmp = tempfile.mkstemp(suffix=".so", dir=PKG, prefix=".libegmla.")
    os.close(fd)
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", INCLUDE, "-I", CSRC, *srcs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        os.unlink(tmp)
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed with exit code {r.returncode}")
    if verbose and r.stderr.strip():
        noise = "packed-fp32-ops' is not a recognized feature"
        msgs = [l for l in r.stderr.splitlines() if noise not in l]
        if msgs:
            sys.stderr.write("\n".join(msgs) + "\n")
    os.replace(tmp, LIB)  # atomic: a loaded old copy stays valid
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    print(build_probe(verbose=True))
