"""Build libmca.so (HIP kernels for gfx950 plus the C ABI) in the package directory,
and beside it libmca_probe.so (issue-cost probes that back the roofline reasoning about
the attention kernels; ``bench.py --issue-probe`` runs them, nothing else loads them).

Usage: ``python -m paper_2201_12854_amd.build_lib`` or ``build()`` from Python.
Compiles every source each time it is called (one hipcc per file, in parallel),
links into ``paper_2201_12854_amd/libmca.so`` and ``libmca_probe.so`` and replaces
the old libraries atomically.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build", "libmca")
LIB = os.path.join(PKG, "libmca.so")
PROBE_LIB = os.path.join(PKG, "libmca_probe.so")
ARCH = "gfx950"

SOURCES = ["k_attention.hip", "k_sample.hip", "k_gather.hip", "k_prepare.hip", "mca_api.cpp"]
PROBE_SOURCES = ["issue_probe.hip"]

CXXFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed-fp32 (v_pk_*_f32) code generation
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in ordinary VGPRs rather than accumulation registers: the attention
    # kernels feed every score to exp2 on the VALU, and a copy out of an accumulation
    # register per score (plus its hazard wait) cost the output pass about a tenth
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP toolchain is required to build libmca")
    return path


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    cmd = [hipcc(), *CXXFLAGS, "-x", "hip", "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = (res.stdout + res.stderr).splitlines()
    noise = "'-packed-fp32-ops' is not a recognized feature"  # host pass of hipcc
    msgs = [l for l in out if noise not in l]
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), flush=True)
    return obj


def _link(objs, lib: str, verbose: bool) -> None:
    tmp = lib + f".tmp{os.getpid()}"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link of {os.path.basename(lib)} failed:\n" + res.stdout + res.stderr)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + PROBE_SOURCES
    with cf.ThreadPoolExecutor(max_workers=4) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    _link(objs[:len(SOURCES)], LIB, verbose)
    _link(objs[len(SOURCES):], PROBE_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
