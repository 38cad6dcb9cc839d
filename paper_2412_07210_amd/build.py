"""Build libedit_outer.so (HIP, gfx950 only) in-tree with hipcc.

    python -m paper_2412_07210_amd.build

Each source compiles to an object under paper_2412_07210_amd/_build/ (in
parallel; the kernels file once per range of worker counts), then links into
paper_2412_07210_amd/libedit_outer.so.
"""
from __future__ import annotations

import os
import re
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIBRARY = os.path.join(PKG, "libedit_outer.so")
SOURCES = ["edit_outer_dispatch.hip", "edit_outer_runtime.hip", "edit_group_kernels.hip", "edit_group_runtime.hip"]
# Compiled once per range of worker counts K (EDIT_K_RANGES in
# edit_outer_internal.h), so its template instantiations build in parallel.
KERNELS = "edit_outer_kernels.hip"
ARCH = "gfx950"

# -packed-fp32-ops off: no v_pk_* fp32 instructions are generated.
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: ROCm is required to build libedit_outer.so")
    return path


def k_ranges() -> list:
    """[(first K, last K)] of the per-range objects of the kernels file."""
    text = open(os.path.join(CSRC, "edit_outer_internal.h")).read()
    line = re.search(r"#define EDIT_K_RANGES\(X\)(.*)", text).group(1)
    return [(int(a), int(b)) for a, b in re.findall(r"X\((\d+), (\d+)\)", line)]


def _jobs() -> list:
    """(source, object name, extra flags) of every compile."""
    jobs = [(src, os.path.splitext(src)[0], []) for src in SOURCES]
    for a, b in k_ranges():
        jobs.append((KERNELS, f"edit_outer_kernels_k{a}_{b}", [f"-DEDIT_K_FIRST={a}", f"-DEDIT_K_LAST={b}"]))
    return jobs


def _compile(job, verbose: bool) -> str:
    src, name, extra = job
    obj = os.path.join(BUILD_DIR, name + ".o")
    cmd = [hipcc(), *HIPCC_FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # The host pass does not know the gfx950 feature flag; that warning is noise.
    noise = "is not a recognized feature for this target"
    msg = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msg}")
    if msg.strip() and verbose:
        print(msg, flush=True)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link the shared library; return its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = _jobs()
    with ThreadPoolExecutor(max_workers=min(len(jobs), os.cpu_count() or 1)) as pool:
        objs = list(pool.map(lambda j: _compile(j, verbose), jobs))
    tmp = LIBRARY + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIBRARY)
    return LIBRARY


if __name__ == "__main__":
    print(build(verbose="-q" not in sys.argv))
