"""Build libsloweave.so (gfx950) in-tree.

    python -m paper_2609_07883_amd.build            # every source
    python -m paper_2609_07883_amd.build --changed  # only sources newer than their objects

HIP sources are compiled with hipcc for gfx950; the host-only C++ sources
with g++.  Objects go to ``_build/`` at the repository root; the shared
library lands next to this file, where the binding loads it.
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
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libsloweave.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
HIP_FLAGS = [f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-I", INCLUDE, "-I", CSRC]
CXX_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-I", INCLUDE, "-I", CSRC,
             "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]


def _sources():
    hip, cxx = [], []
    for f in sorted(os.listdir(CSRC)):
        p = os.path.join(CSRC, f)
        if f.endswith(".hip"):
            hip.append(p)
        elif f.endswith(".cpp"):
            cxx.append(p)
    return hip, cxx


def _newest_header() -> float:
    hs = [os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")]
    hs += [os.path.join(INCLUDE, f) for f in os.listdir(INCLUDE) if f.endswith(".h")]
    return max(os.path.getmtime(h) for h in hs)


def _compile(src: str, changed_only: bool = False) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    if changed_only and os.path.exists(obj) and \
            os.path.getmtime(obj) > max(os.path.getmtime(src), _newest_header()):
        return obj
    if src.endswith(".hip"):
        cmd = [HIPCC, *HIP_FLAGS, "-c", src, "-o", obj]
    else:
        cmd = ["g++", *CXX_FLAGS, "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    # the host pass of hipcc warns about the device-only feature flag; keep other warnings
    warn = [ln for ln in r.stderr.splitlines() if ln.strip() and "packed-fp32-ops" not in ln]
    if warn:
        sys.stderr.write("\n".join(warn) + "\n")
    return obj


def build_library(jobs: int = 8, changed_only: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    hip, cxx = _sources()
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda f: _compile(f, changed_only), hip + cxx))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    shutil.move(tmp, LIB)
    return LIB


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("-j", type=int, default=8)
    ap.add_argument("--changed", action="store_true", help="compile only sources newer than their objects")
    args = ap.parse_args()
    print(build_library(args.j, args.changed))


if __name__ == "__main__":
    main()
