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

# Packed fp32 ALU instructions are disabled for all device code.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-Wno-unused-command-line-argument"]

# The matrix-core kernels run with the IEEE mode bit clear and are compiled
# without NaN semantics: no result depends on NaN propagation (masked scores
# are -inf, reads past valid rows never happen), and the compiler then emits
# plain v_max/v_max3 without a quieting v_max(x, x) before each operand, a
# tenth of their vector instructions.  The vector-ALU kernels compile to
# slower code with the same flags, so they keep the defaults.
SOURCE_FLAGS = {"split_mfma.hip": ["-fno-honor-nans", "-mno-amdgpu-ieee"]}


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
    for name in sorted(SOURCE_FLAGS):
        h.update((name + " " + " ".join(SOURCE_FLAGS[name])).encode())
    return h.hexdigest()


def _run(cmd, verbose):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    if verbose:
        print(" ".join(cmd))
        print(r.stderr)


def build_library(verbose: bool = False, extra_flags=()) -> str:
    """Compiles each translation unit with its flags, then links them."""
    out_dir = os.path.dirname(LIBRARY)
    os.makedirs(out_dir, exist_ok=True)
    objs = []
    for src in sources():
        name = os.path.basename(src)
        obj = os.path.join(out_dir, name + ".o")
        _run([HIPCC, *HIP_FLAGS, *SOURCE_FLAGS.get(name, []), *extra_flags, "-I", INCLUDE, "-I", CSRC,
              "-c", src, "-o", obj], verbose)
        objs.append(obj)
    tmp = LIBRARY + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build_library(verbose=True))
