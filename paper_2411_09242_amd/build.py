"""Build the two shared libraries behind include/fluid.h, in-tree.

  lib/libfluid.so       host planners + HIP kernels for gfx950 (hipcc)
  lib/libfluid_host.so  host planners only (g++); GPU entry points return
                        FLUID_E_UNSUPPORTED.  Used by CPU-only tests.

Usage: python -m paper_2411_09242_amd.build [--host-only] [--jobs N]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIBDIR = os.path.join(PKG, "lib")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

CXXFLAGS = ["-std=c++17", "-O2", "-fPIC", "-Wall", "-Wno-unused-function", f"-I{INCLUDE}"]
# Packed fp32 VALU instructions are disabled for all device code: the
# compiler would otherwise form them from plain fp32 code.
HIPFLAGS = ["-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}", f"-I{INCLUDE}",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-result"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def _obj(src, tag):
    rel = os.path.relpath(src, CSRC).replace(os.sep, "_")
    return os.path.join(BUILD, tag, rel + ".o")


def _compile(job):
    src, obj, cmd = job
    if os.path.exists(obj) and os.path.getmtime(obj) >= _newest_dep(src):
        return obj
    os.makedirs(os.path.dirname(obj), exist_ok=True)
    _run(cmd + ["-c", src, "-o", obj])
    return obj


_HEADERS = None


def _newest_dep(src):
    global _HEADERS
    if _HEADERS is None:
        hs = glob.glob(os.path.join(CSRC, "**", "*.h"), recursive=True)
        hs.append(os.path.join(INCLUDE, "fluid.h"))
        _HEADERS = max(os.path.getmtime(h) for h in hs)
    return max(os.path.getmtime(src), _HEADERS, os.path.getmtime(__file__))


def build(host_only=False, jobs=None, force=False):
    if force and os.path.isdir(BUILD):
        shutil.rmtree(BUILD)
    os.makedirs(LIBDIR, exist_ok=True)
    host_srcs = sorted(glob.glob(os.path.join(CSRC, "host", "*.cpp")))
    core = [s for s in host_srcs if not s.endswith("host_stubs.cpp")]
    stub = [s for s in host_srcs if s.endswith("host_stubs.cpp")]
    hip_srcs = sorted(glob.glob(os.path.join(CSRC, "gpu", "*.hip")))
    jobs_list = [(s, _obj(s, "host"), ["g++"] + CXXFLAGS) for s in core + stub]
    if not host_only:
        jobs_list += [(s, _obj(s, "gpu"), [HIPCC] + HIPFLAGS) for s in hip_srcs]
    n = jobs or min(16, os.cpu_count() or 4)
    with cf.ThreadPoolExecutor(max_workers=n) as ex:
        list(ex.map(_compile, jobs_list))
    host_lib = os.path.join(LIBDIR, "libfluid_host.so")
    _run(["g++", "-shared", "-o", host_lib + ".tmp"] + [_obj(s, "host") for s in core + stub])
    os.replace(host_lib + ".tmp", host_lib)
    if host_only:
        return [host_lib]
    gpu_lib = os.path.join(LIBDIR, "libfluid.so")
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", gpu_lib + ".tmp"]
         + [_obj(s, "host") for s in core] + [_obj(s, "gpu") for s in hip_srcs])
    os.replace(gpu_lib + ".tmp", gpu_lib)
    return [host_lib, gpu_lib]


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--host-only", action="store_true")
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("--force", action="store_true")
    a = ap.parse_args(argv)
    for p in build(a.host_only, a.jobs, a.force):
        print(p)


if __name__ == "__main__":
    sys.exit(main())
