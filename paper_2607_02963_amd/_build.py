"""Builds libpdec.so (the HIP kernels and the C ABI) in-tree for gfx950."""
from __future__ import annotations

import hashlib
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "_build", "libpdec.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed fp32 ALU instructions are disabled for all device code.  The
# kernels run with the IEEE mode bit clear and are compiled without NaN
# semantics: no result depends on NaN propagation (masked scores are -inf,
# reads past valid rows never happen), and the compiler then emits plain
# v_max/v_max3 without a quieting v_max(x, x) before each operand, which
# is about a tenth of the split kernels' vector instructions.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-fno-honor-nans", "-mno-amdgpu-ieee",
             "-Wno-unused-command-line-argument"]


def sources():
    return [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC)) if f.endswith(".hip")]


def source_digest() -> str:
    """sha256 over the kernel sources, the public header and the compile
    flags: names the build a stored profile was measured with."""
    h = hashlib.sha256()
    for d in (CSRC, INCLUDE):
        for f in sorted(os.listdir(d)):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    h.update(" ".join(HIP_FLAGS).encode())
    return h.hexdigest()


def build_library(verbose: bool = False, extra_flags=()) -> str:
    os.makedirs(os.path.dirname(LIBRARY), exist_ok=True)
    tmp = LIBRARY + ".tmp"
    cmd = [HIPCC, *HIP_FLAGS, *extra_flags, "-I", INCLUDE, "-I", CSRC, *sources(), "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    if verbose:
        print(" ".join(cmd))
        print(r.stderr)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build_library(verbose=True))
