"""Build libhla.so for gfx950 with hipcc, in-tree.

    python -m paper_2511_05832_amd.build [--debug] [-j N]

Compiles every source in csrc/ to an object under _build/ and links
paper_2511_05832_amd/libhla.so. Always recompiles (the build is a few seconds
per file); the objects are compiled in parallel.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhla.so")
ARCH = "gfx950"

SOURCES = ["hla_api.cpp", "hilbert.hip", "permute.hip", "blockmask.hip",
           "attn_bf16.hip", "attn_f32.hip", "attn_bwd_bf16.hip",
           "attn_bwd_f32.hip", "proj.hip"]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP toolchain is required to build libhla")
    return path


def common_flags(debug: bool):
    flags = [f"--offload-arch={ARCH}", "-std=c++17", "-fPIC", "-I", INCLUDE, "-I", CSRC,
             # keep the compiler from forming packed fp32 ops on its own
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             # matrix-core accumulators in ordinary VGPRs: the softmax and rescale
             # work on them with VALU ops, which cannot read AGPRs
             "-mllvm", "-amdgpu-mfma-vgpr-form=1",
             "-Wall", "-Wno-unused-result", "-Wno-unused-variable",
             "-Wno-unknown-pragmas"]
    flags += ["-O1", "-g"] if debug else ["-O3"]
    return flags


def compile_one(src: str, debug: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc()] + common_flags(debug) + ["-c", os.path.join(CSRC, src), "-o", obj]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{out}")
    if out.strip():
        print(out, file=sys.stderr)
    return obj


def build(debug: bool = False, jobs: int = 0) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = jobs or min(len(SOURCES), os.cpu_count() or 4)
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda s: compile_one(s, debug), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"linking libhla.so failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    return LIB


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--debug", action="store_true")
    ap.add_argument("-j", type=int, default=0)
    args = ap.parse_args()
    print(build(args.debug, args.j))


if __name__ == "__main__":
    main()
