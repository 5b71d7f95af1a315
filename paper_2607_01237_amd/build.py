"""Builds libkara.so (HIP for gfx950) in this package directory.

    python -m paper_2607_01237_amd.build

Each source compiles to its own object in _build/ (in parallel), then hipcc
links the shared library.  Always rebuilds.
"""

from __future__ import annotations

import glob
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
LIB = os.path.join(PKG, "libkara.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    # packed fp32 VALU forms stay off: the compiler would otherwise emit them from ordinary float code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


# Per-file options.  Selection: a smaller limit on promoting private arrays
# to vectors leaves the 8-position instance's per-thread arrays as separate
# registers (56 VGPRs instead of 126, no scratch either way).
FILE_FLAGS = {
    "kara_select.hip": ["-mllvm", "-amdgpu-promote-alloca-to-vector-limit=256"],
    # scoring: MFMA results in ordinary VGPRs, read directly by the vector
    # instructions; the accumulation registers hold the single-sweep
    # kernel's stored weights
    "kara_score.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}
# rocBLAS runs the recompute pass's plain matrix products
LINK_LIBS = ["-L/opt/rocm/lib", "-lrocblas"]


def source_hash() -> str:
    """SHA-256 over every source, header and compile option the library is
    built from.  The build bakes it into libkara.so (kara_source_hash) and the
    binding compares it at load time, so a library built from other sources
    is refused instead of silently tested."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(CSRC, "*")) + glob.glob(os.path.join(INCLUDE, "*.h")))
    for path in files:
        if os.path.isfile(path):
            h.update(os.path.basename(path).encode())
            with open(path, "rb") as f:
                h.update(f.read())
    # options with the checkout's location taken out, so the same tree hashes
    # the same wherever it sits
    flags = [f.replace(ROOT, "<root>") for f in FLAGS]
    h.update(repr((ARCH, flags, sorted(FILE_FLAGS.items()), LINK_LIBS)).encode())
    return h.hexdigest()


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in r.stdout.splitlines() if "is not a recognized feature" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))
    objs = [os.path.join(BUILD, os.path.basename(s) + ".o") for s in srcs]

    digest = source_hash()

    def compile_one(pair):
        src, obj = pair
        extra = [f'-DKARA_SOURCE_HASH="{digest}"'] if os.path.basename(src) == "kara_api.cpp" else []
        return _run([HIPCC, *FLAGS, *FILE_FLAGS.get(os.path.basename(src), []), *extra, "-c", src, "-o", obj])

    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        outs = list(ex.map(compile_one, zip(srcs, objs)))
    tmp = LIB + ".tmp"
    outs.append(_run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, *LINK_LIBS, "-o", tmp]))
    os.replace(tmp, LIB)
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
