"""Build the gfx950 HIP library (librac.so) in-tree with hipcc.

Flags: -ffp-contract=off keeps every multiply and add separately rounded (the
codec's arithmetic is defined operation by operation); packed fp32 ops are
disabled; divisions stay correctly rounded (hipcc's default).

The device assembly is also generated and scanned for a known miscompile
(see isa_check.py); a hit fails the build.
"""
from __future__ import annotations

import os
import subprocess
import sys

try:
    from . import isa_check
except ImportError:  # run as a script
    import isa_check

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "rac.hip")
HOST_SRC = os.path.join(HERE, "csrc", "spans.cpp")   # host-only C++ (reference selection)
PRED_SRC = os.path.join(HERE, "csrc", "predictor.hip")  # decode-phase reference predictor
INC = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "lib", "librac.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-ffp-contract=off", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function"]


def build(verbose: bool = True) -> str:
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *FLAGS, "-I", INC, "-o", tmp, SRC, PRED_SRC, HOST_SRC]
    asm = LIB + ".s"
    dev = [HIPCC, *[f for f in FLAGS if f not in ("-fPIC", "-shared")], "--cuda-device-only", "-S",
           "-I", INC, "-o", asm, SRC]
    if verbose:
        print(" ".join(cmd), flush=True)
    # the library and the device assembly that is scanned are independent
    # compiles: run them side by side
    procs = [subprocess.Popen(cmd), subprocess.Popen(dev)]
    codes = [p.wait() for p in procs]
    if any(codes):
        for f in (tmp, asm):
            if os.path.exists(f):
                os.remove(f)
        raise subprocess.CalledProcessError(next(c for c in codes if c), cmd if codes[0] else dev)
    bad = isa_check.scan(open(asm).read())
    os.remove(asm)
    if bad:
        os.remove(tmp)
        raise RuntimeError("miscompiled SCC use in librac:\n" + "\n".join(bad))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
