"""Build the HIP library for gfx950.

    python paper_2102_08550_amd/build.py

Produces, in ``paper_2102_08550_amd/_lib/``:
  liboscars.so        the C-ABI library (HIP kernels + host runtime), gfx950
  liboscars_host.so   host-only parts (Algorithm 1, shards, sampler, weights),
                      plain g++ build used by CPU tests
  liboscars_host_san.so  the same host-only parts with AddressSanitizer and
                      UndefinedBehaviorSanitizer (loaded by a CPU test under
                      LD_PRELOAD of libasan)
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "_lib")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    os.makedirs(OUT, exist_ok=True)
    objdir = os.path.join(OUT, "obj")
    os.makedirs(objdir, exist_ok=True)
    objs = []
    for src in ("kernels.hip", "conv_kernels.hip", "runtime.hip"):
        obj = os.path.join(objdir, src + ".o")
        _run([HIPCC, *HIP_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    host_obj = os.path.join(objdir, "host_logic.o")
    _run(["g++", *HOST_FLAGS, "-c", os.path.join(CSRC, "host_logic.cpp"), "-o", host_obj])
    objs.append(host_obj)
    lib = os.path.join(OUT, "liboscars.so")
    tmp = lib + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, lib)
    # host-only libraries for CPU tests
    _run(["g++", *HOST_FLAGS, "-shared", os.path.join(CSRC, "host_logic.cpp"), "-o",
          os.path.join(OUT, "liboscars_host.so")])
    try:
        _run(["g++", *HOST_FLAGS, "-g", "-fno-omit-frame-pointer",
              "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-shared",
              os.path.join(CSRC, "host_logic.cpp"), "-o",
              os.path.join(OUT, "liboscars_host_san.so")])
    except RuntimeError as e:  # sanitizer runtime missing: the CPU test skips
        if verbose:
            print(e)
    shutil.rmtree(objdir, ignore_errors=True)
    if verbose:
        print("built", lib)
    return lib


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
