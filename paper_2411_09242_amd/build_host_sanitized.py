"""Build the host-only library with AddressSanitizer and UndefinedBehavior-
Sanitizer (g++, CPU code only) into _build/san/lib/libfluid_host.so.

The CPU tests can then run against it (FLUID_LIBDIR=<that directory>, with
the ASan runtime preloaded into the interpreter): every planner, table
loader and launch-preparation path is exercised with bounds, use-after-free
and undefined-behaviour checks, and any report aborts the test process.

Usage: python -m paper_2411_09242_amd.build_host_sanitized
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build", "san")
LIBDIR = os.path.join(PKG, "_build", "san", "lib")
SANFLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
CXXFLAGS = ["-std=c++17", "-O1", "-g", "-fPIC", "-Wall", "-Wno-unused-function", f"-I{INCLUDE}"] + SANFLAGS


def runtime_library():
    """Path of the ASan runtime the library links against (to preload)."""
    r = subprocess.run(["g++", "-print-file-name=libasan.so"], stdout=subprocess.PIPE, text=True, check=True)
    return r.stdout.strip()


def _compile(src):
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    deps = glob.glob(os.path.join(CSRC, "host", "*.h")) + [os.path.join(INCLUDE, "fluid.h"), src]
    if not (os.path.exists(obj) and os.path.getmtime(obj) >= max(os.path.getmtime(d) for d in deps)):
        subprocess.run(["g++"] + CXXFLAGS + ["-c", src, "-o", obj], check=True)
    return obj


def build():
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "host", "*.cpp")))
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, srcs))
    lib = os.path.join(LIBDIR, "libfluid_host.so")
    subprocess.run(["g++", "-shared"] + SANFLAGS + ["-o", lib + ".tmp"] + objs, check=True)
    os.replace(lib + ".tmp", lib)
    return lib


if __name__ == "__main__":
    print(build())
    sys.exit(0)
