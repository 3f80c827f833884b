"""Build libsparse_linear.so in-tree for gfx950.

    python -m paper_2211_07715_amd.build

The HIP kernels are compiled with hipcc for gfx950 only (packed-fp32 VALU
instructions disabled); the host packer and the C-ABI layer are plain C++.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libsparse_linear.so")
PROBE_LIB = os.path.join(HERE, "libsl_probe.so")
BUILD_DIR = os.path.join(ROOT, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HOST_SOURCES = ["api.cpp", "pack.cpp", "gelu_table.cpp"]
HIP_SOURCES = ["kernels.hip", "kernels_direct.hip", "kernels_panel.hip", "kernels_split.hip"]
# the benchmark's measurement probes (copy bandwidth, matrix-instruction
# throughput): a library of their own, not linked into the layer's
PROBE_SOURCES = ["probe.hip"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


def build(verbose: bool = False) -> str:
    """Compile every source (in parallel) and link the shared library."""
    from concurrent.futures import ThreadPoolExecutor

    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        jobs.append((["g++", "-std=c++17", "-O2", "-ffp-contract=off", "-fPIC", "-Wall", "-Wextra", "-I", INCLUDE,
                      "-c", os.path.join(CSRC, src), "-o", obj], obj))
    for src in HIP_SOURCES + PROBE_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        jobs.append(([HIPCC, f"--offload-arch={ARCH}", "-std=c++17", "-O3", "-fPIC", "-Wall", *DEVICE_FLAGS,
                      "-I", INCLUDE, "-c", os.path.join(CSRC, src), "-o", obj], obj))
    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as ex:
        for f in [ex.submit(_run, cmd, verbose) for cmd, _ in jobs]:
            f.result()
    probe_objs = [os.path.join(BUILD_DIR, src + ".o") for src in PROBE_SOURCES]
    objs = [obj for _, obj in jobs if obj not in probe_objs]
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp], verbose)
    os.replace(tmp, LIB)
    tmp = PROBE_LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *probe_objs, "-o", tmp], verbose)
    os.replace(tmp, PROBE_LIB)
    return LIB


def clean():
    shutil.rmtree(BUILD_DIR, ignore_errors=True)
    for lib in (LIB, PROBE_LIB):
        if os.path.exists(lib):
            os.remove(lib)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
