"""Build libluna.so (HIP kernels for gfx950 + the C ABI host code) in-tree.

Usage: python -m paper_2512_08061_amd.build  (or __graft_entry__.build()).
Each source is compiled to an object under paper_2512_08061_amd/_build/ in
parallel, then linked into paper_2512_08061_amd/libluna.so.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys
import time

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libluna.so")

SOURCES = ["luna_prepare.hip", "luna_featuremap.hip", "luna_noncausal.hip", "luna_causal.hip", "luna_stream.hip",
           "luna_variants.hip", "luna_variants_bf16.hip", "luna_distill.hip",
           "luna_backward.hip", "luna_api.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-variable",
    "-Wno-unused-function",
    # packed fp32 VALU instructions are kept out of all device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


def _compile(src: str, extra: list[str]) -> tuple[str, float]:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, "-x", "hip", *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    t0 = time.time()
    p = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (p.stdout + p.stderr).splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"compiling {src} failed:\n{' '.join(cmd)}\n{msgs}")
    if msgs.strip():
        print(msgs, file=sys.stderr)
    return obj, time.time() - t0


def build(verbose: bool = True, extra: list[str] | None = None, jobs: int | None = None) -> str:
    os.makedirs(BUILD, exist_ok=True)
    extra = list(extra or [])
    jobs = jobs or min(len(SOURCES), max(1, len(os.sched_getaffinity(0))))
    t0 = time.time()
    with cf.ThreadPoolExecutor(jobs) as ex:
        futs = {ex.submit(_compile, s, extra): s for s in SOURCES}
        objs = {}
        for f in cf.as_completed(futs):
            obj, dt = f.result()
            objs[futs[f]] = obj
            if verbose:
                print(f"  compiled {futs[f]} in {dt:.1f}s", file=sys.stderr)
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *[objs[s] for s in SOURCES]]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"linking libluna.so failed:\n{' '.join(cmd)}\n{p.stdout}{p.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} in {time.time() - t0:.1f}s", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
