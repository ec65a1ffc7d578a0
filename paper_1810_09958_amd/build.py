"""Build libisam.so (gfx950) in-tree with hipcc.

Every HIP source is compiled for gfx950 only, with packed-fp32 instruction
selection disabled, then linked into ``paper_1810_09958_amd/libisam.so``.
Run ``python -m paper_1810_09958_amd.build`` (or ``__graft_entry__.build()``).
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libisam.so")
SOURCES = ["api.cpp", "launch_cache.cpp", "gemm.hip", "gemm_bf16.hip", "gemm_f32.hip", "gemm_dma.hip", "gemm_dma_sk.hip", "gemm_small.hip", "gemm_stream.hip", "pack.hip", "skinny.hip", "dwconv.hip", "dwsep_fused.hip", "dwsep_fused_f32.hip", "gru.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def flags():
    return ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(HERE, "..", "include")]


def build(jobs: int = 8, verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    cc = hipcc()
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        objs.append(obj)
        cmd = [cc, *flags(), "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
        while len([p for _, p in procs if p.poll() is None]) >= jobs:
            procs[0][1].wait() if procs[0][1].poll() is None else None
            break
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = "\n".join(l for l in out.decode(errors="replace").splitlines()
                         if "packed-fp32-ops" not in l)
        if p.returncode != 0:
            failed.append((src, text))
        elif verbose and text.strip():
            print(text)
    if failed:
        msg = "\n".join(f"--- {s} ---\n{t}" for s, t in failed)
        raise RuntimeError(f"hipcc failed:\n{msg}")
    tmp = LIB + ".tmp"
    subprocess.run([cc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs], check=True,
                   stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    os.replace(tmp, LIB)
    return LIB


SAN_LIB = os.path.join(BUILD, "libisam_san.so")


def build_sanitized() -> str:
    """A copy of the library whose host code (argument validation, planning and dispatch in
    api.cpp) is built with g++ under AddressSanitizer and UndefinedBehaviorSanitizer, linked
    with the device objects of the regular build.  For the CPU test tier: load it with gcc's
    libasan and libubsan preloaded and ISAM_LIB pointing at it."""
    if not all(os.path.exists(os.path.join(BUILD, src + ".o")) for src in SOURCES):
        build()
    obj = os.path.join(BUILD, "api.cpp.san.o")
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(rocm, "include"), "-I", os.path.join(HERE, "..", "include"), *san,
                    "-c", os.path.join(CSRC, "api.cpp"), "-o", obj], check=True)
    objs = [obj] + [os.path.join(BUILD, src + ".o") for src in SOURCES if src != "api.cpp"]
    tmp = SAN_LIB + ".tmp"
    subprocess.run(["g++", "-shared", "-o", tmp, *objs, "-L", os.path.join(rocm, "lib"),
                    "-Wl,-rpath," + os.path.join(rocm, "lib"), "-lamdhip64", *san], check=True)
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitized" in sys.argv:
        print(build_sanitized())
    else:
        print(build(verbose="-v" in sys.argv))
