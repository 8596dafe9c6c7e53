"""Build the HIP library libmasq.so in-tree for gfx950.

    python -m paper_2603_04800_amd.build [--remarks]

The library is compiled with hipcc (ROCm >= 7) for gfx950 only, without FP
contraction and with correctly rounded fp32 division and square root (both
are part of the bit-exact contract of masq.h).  Packed fp32 arithmetic is
disabled for the device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "libmasq.so")
SOURCES = ("masq_kernels.hip", "masq_api.hip", "masq_calib.hip", "masq_linalg.hip")
# the benchmark's peak probes, a library of their own (not part of the layer)
PROBE_SOURCES = ("masq_probe.hip",)
PROBE_LIB = os.path.join(LIBDIR, "libmasq_probe.so")


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libmasq.so)")


def compile_flags(remarks: bool = False):
    flags = [
        "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
        "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC,
    ]
    if remarks:
        flags.append("-Rpass-analysis=kernel-resource-usage")
    return flags


def build(remarks: bool = False, verbose: bool = True) -> str:
    _build_lib(SOURCES, LIB, remarks, verbose)
    _build_lib(PROBE_SOURCES, PROBE_LIB, remarks, verbose)
    return LIB


def _build_lib(sources, lib, remarks: bool, verbose: bool) -> str:
    os.makedirs(LIBDIR, exist_ok=True)
    objs = []
    for src in sources:
        obj = os.path.join(LIBDIR, src.replace(".hip", ".o"))
        cmd = [hipcc(), *compile_flags(remarks), "-c", os.path.join(CSRC, src), "-o", obj]
        res = subprocess.run(cmd, capture_output=True, text=True)
        out = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                        if "packed-fp32-ops" not in l)
        if verbose and out.strip():
            print(out)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{out}")
        objs.append(obj)
    tmp = lib + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}{res.stderr}")
    os.replace(tmp, lib)
    return lib


SANITIZED_LIB = os.path.join(LIBDIR, "libmasq_sanitized.so")


def build_sanitized(verbose: bool = False) -> str:
    """libmasq_sanitized.so: the library with the host code of its entry
    points (argument validation, workspace planning, dispatch: masq_api.hip,
    masq_calib.hip, masq_linalg.hip) built with AddressSanitizer and UndefinedBehaviorSanitizer;
    device code is not instrumented.  Reuses the kernel object of build()
    when it is present."""
    os.makedirs(LIBDIR, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]
    objs = []
    for src in SOURCES:
        obj = os.path.join(LIBDIR, src.replace(".hip", ".o"))
        if src in ("masq_api.hip", "masq_calib.hip", "masq_linalg.hip"):
            obj = os.path.join(LIBDIR, src.replace(".hip", "_sanitized.o"))
            flags = [*compile_flags(), *san]
        elif os.path.exists(obj):
            objs.append(obj)
            continue
        else:
            flags = compile_flags()
        res = subprocess.run([hipcc(), *flags, "-c", os.path.join(CSRC, src), "-o", obj],
                             capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"hipcc failed for {src}:\n{res.stdout}{res.stderr}")
        objs.append(obj)
    res = subprocess.run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *san, *objs, "-o",
                          SANITIZED_LIB], capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}{res.stderr}")
    return SANITIZED_LIB


if __name__ == "__main__":
    print(build(remarks="--remarks" in sys.argv))
