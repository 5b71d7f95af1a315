"""Builds a host-sanitized copy of libkara.so for the CPU tests.

    python -m paper_2607_01237_amd.build_sanitized

Every source is compiled as for the product library, with AddressSanitizer
and UndefinedBehaviorSanitizer on the host side only (-Xarch_host; the gfx950
code is unchanged), into _build_san/libkara_san.so.  The library is linked
without the sanitizer runtime: a process loads clang's shared ASan runtime
first (LD_PRELOAD, as tests/test_host_sanitizers.py does), and every
undefined-behaviour report aborts.  Only host code runs under it: the
argument checks of the C ABI and the scheduler runtime, no kernel.
"""

from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

from . import build as _b

BUILD = os.path.join(_b.PKG, "_build_san")
LIB = os.path.join(BUILD, "libkara_san.so")
HOST_SANITIZE = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
                 "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"]


def runtime() -> str:
    """Path of clang's shared ASan runtime (it carries the UBSan handlers)."""
    out = subprocess.run([_b.HIPCC, "-print-file-name=libclang_rt.asan-x86_64.so"], stdout=subprocess.PIPE,
                         stderr=subprocess.DEVNULL, text=True).stdout.strip()
    if out and os.path.exists(out):
        return out
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang's shared ASan runtime was not found")
    return hits[-1]


def build() -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(_b.CSRC, "*.hip")) + glob.glob(os.path.join(_b.CSRC, "*.cpp")))
    objs = [os.path.join(BUILD, os.path.basename(s) + ".o") for s in srcs]
    digest = _b.source_hash()

    def compile_one(pair):
        src, obj = pair
        extra = [f'-DKARA_SOURCE_HASH="{digest}"'] if os.path.basename(src) == "kara_api.cpp" else []
        return _b._run([_b.HIPCC, *_b.FLAGS, *_b.FILE_FLAGS.get(os.path.basename(src), []), *HOST_SANITIZE,
                        *extra, "-c", src, "-o", obj])

    with ThreadPoolExecutor(min(8, len(srcs))) as ex:
        list(ex.map(compile_one, zip(srcs, objs)))
    tmp = LIB + ".tmp"
    _b._run([_b.HIPCC, f"--offload-arch={_b.ARCH}", "-shared", "-fPIC", *objs, *_b.LINK_LIBS, "-o", tmp])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
    if "-v" in sys.argv:
        print(runtime())
