"""Build the gfx950 device library and the host-only bookkeeping library.

    python -m paper_2609_36899_amd.build

produces, next to this file:
  libpdec.so       -- HIP kernels + C ABI (include/pdec.h), built by hipcc for gfx950
  libpdec_host.so  -- page pool, attention planner and pacing only, built by g++ (CPU tests)

    python -m paper_2609_36899_amd.build --sanitize

builds libpdec_host_san.so, the host library under AddressSanitizer and
UndefinedBehaviorSanitizer (tests/test_sanitizers.py runs the host tests on it).
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
ROOT = os.path.dirname(PKG)
BUILD = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_SOURCES = ["attention.hip", "attention_prefill.hip", "gemm.hip", "pointwise.hip", "kvcopy.hip",
               "sample.hip", "engine.cpp", "pagepool.cpp", "pacing.cpp"]
HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # Packed fp32 VALU ops are kept out of the device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    f"-I{os.path.join(ROOT, 'include')}",
]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(line for line in r.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build_device(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    cmds = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmds.append([HIPCC, *HIP_FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(cmds))) as ex:
        for out in ex.map(_run, cmds):
            if verbose and out.strip():
                print(out)
    lib = os.path.join(PKG, "libpdec.so")
    tmp = lib + ".tmp"
    _run([HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp])
    os.replace(tmp, lib)
    return lib


HOST_SOURCES = ["pagepool.cpp", "pacing.cpp", "host_capi.cpp"]
# The sanitizer build of the host library: AddressSanitizer and
# UndefinedBehaviorSanitizer, every finding fatal.  Load it with the two
# runtimes preloaded (SANITIZER_RUNTIMES) and ASAN_OPTIONS=detect_leaks=0
# (the interpreter's own allocations are not ours).
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all"]
SANITIZER_RUNTIMES = ("libasan.so", "libubsan.so")


def build_host(sanitize: bool = False) -> str:
    """libpdec_host.so (g++ -O2), or with sanitize=True libpdec_host_san.so."""
    lib = os.path.join(PKG, "libpdec_host_san.so" if sanitize else "libpdec_host.so")
    tmp = lib + ".tmp"
    flags = SANITIZE_FLAGS if sanitize else ["-O2"]
    _run(["g++", *flags, "-std=c++17", "-fPIC", "-shared", "-Wall", "-Werror",
          f"-I{os.path.join(ROOT, 'include')}",
          *[os.path.join(CSRC, f) for f in HOST_SOURCES], "-o", tmp])
    os.replace(tmp, lib)
    return lib


def sanitizer_preload() -> str:
    """LD_PRELOAD value that loads the sanitizer runtimes of g++."""
    paths = []
    for name in SANITIZER_RUNTIMES:
        r = subprocess.run(["g++", f"-print-file-name={name}"], stdout=subprocess.PIPE,
                           text=True, check=True)
        paths.append(r.stdout.strip())
    return ":".join(paths)


def build_all(verbose: bool = False):
    return build_host(), build_device(verbose)


if __name__ == "__main__":
    if "--sanitize" in sys.argv:
        print(build_host(sanitize=True))
    else:
        for p in build_all(verbose="-v" in sys.argv):
            print(p)
