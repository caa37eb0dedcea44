"""Build the HIP library in-tree for gfx950.

    python -m paper_1904_12380_amd.build

Produces paper_1904_12380_amd/lib/libsoftmax_mi355x.so from csrc/ with
hipcc.  Compiles every time it is called.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIBDIR = os.path.join(PKG, "lib")
LIB = os.path.join(LIBDIR, "libsoftmax_mi355x.so")
SOURCES = [os.path.join(CSRC, "softmax_api.hip"), os.path.join(CSRC, "attention_api.hip")]

ARCH = "gfx950"
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-fvisibility=hidden",
    # Rounding steps of the two-sum in the exp argument must stay as written.
    "-ffp-contract=off",
    # No packed fp32 instructions in any generated code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    return subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)


def _finish(proc, verbose):
    out, _ = proc.communicate()
    if proc.returncode != 0:
        sys.stderr.write(out)
        raise RuntimeError(f"hipcc failed with exit code {proc.returncode}")
    noise = "packed-fp32-ops"  # the host pass does not know the feature
    for line in out.splitlines():
        if verbose and noise not in line and line.strip():
            print(line)


def build(verbose: bool = False) -> str:
    """Compile each source to an object (in parallel), then link the .so."""
    os.makedirs(LIBDIR, exist_ok=True)
    tag = f".tmp{os.getpid()}"
    objs = [os.path.join(LIBDIR, os.path.basename(src) + tag + ".o") for src in SOURCES]
    compile_flags = [f for f in HIPCC_FLAGS if f != "-shared"]
    procs = [_run([hipcc(), *compile_flags, "-I", os.path.join(ROOT, "include"), "-c", src,
                   "-o", obj], verbose) for src, obj in zip(SOURCES, objs)]
    try:
        for proc in procs:
            _finish(proc, verbose)
        tmp = LIB + tag
        _finish(_run([hipcc(), *HIPCC_FLAGS, *objs, "-o", tmp], verbose), verbose)
        os.replace(tmp, LIB)
    finally:
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
