"""Build libstepprune.so (and the benchmark's LDS probe, libstepprune_probe.so)
for gfx950 with hipcc (in-tree, next to this file).

    python -m paper_2609_13804_amd.build [--jobs N] [--verbose]
"""
import argparse
import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libstepprune.so")
PROBE_LIB = os.path.join(HERE, "libstepprune_probe.so")
PROBE_SOURCE = "probe.hip"
BUILD_DIR = os.path.join(ROOT, "_build")

SOURCES = ["api.hip", "gemm.hip", "select.hip", "text.hip", "compact.hip", "denoise.hip",
           "encode.hip"]
# The selection recurrence keeps each column's history in vector registers; let
# alloca promotion use the whole VGPR budget instead of a quarter of it.
EXTRA_FLAGS = {"select.hip": ["-mllvm", "-amdgpu-promote-alloca-to-vector-vgpr-ratio=1"]}
ARCH = "gfx950"
# roctx ranges around the entry points (rocprofiler-sdk's marker library)
LINK_LIBS = ["-lrocprofiler-sdk-roctx"]
# Packed fp32 ALU ops are disabled for every translation unit.
HIPCC_FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", INCLUDE, "-I", CSRC, "-Wall", "-Wno-unused-function"]


def _hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; ROCm is required to build libstepprune")
    return path


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in r.stderr.splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{err}")
    if verbose and err.strip():
        print(err)


def build(jobs: int = 8, verbose: bool = False) -> str:
    """Compile every translation unit and link libstepprune.so; returns its path."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(BUILD_DIR, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([hipcc, *HIPCC_FLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src),
                     "-o", obj])
    with concurrent.futures.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        list(ex.map(lambda c: _run(c, verbose), cmds))
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs, *LINK_LIBS],
         verbose)
    os.replace(tmp, LIB)
    # the benchmark's LDS bandwidth probe, a library of its own
    tmp = PROBE_LIB + ".tmp"
    _run([hipcc, *HIPCC_FLAGS, "-shared", "-o", tmp, os.path.join(CSRC, PROBE_SOURCE)], verbose)
    os.replace(tmp, PROBE_LIB)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=8)
    ap.add_argument("--verbose", action="store_true")
    args = ap.parse_args(argv)
    print(build(args.jobs, args.verbose))


if __name__ == "__main__":
    sys.exit(main())
