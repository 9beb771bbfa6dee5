"""Build libprecache.so (the C-ABI library) for gfx950 with hipcc, in-tree.

Usage: ``python -m paper_2609_34054_amd.build`` or ``build()`` from Python.
Every call recompiles all sources (objects go to ``_build/``), then links
``paper_2609_34054_amd/libprecache.so`` and its checked twin
``libprecache_checked.so`` (the same kernels; the ABI layer compiled with
``PRC_DEVICE_CHECKS=1`` checks device-resident kv_len and positions).
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
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB_PATH = os.path.join(PKG, "libprecache.so")
CHECKED_LIB_PATH = os.path.join(PKG, "libprecache_checked.so")

SOURCES = [
    "abi.cpp",
    "precompute_gemm.hip",
    "lrsa_decode.hip",
    "lrsa_prefill.hip",
    "materialize.hip",
    "stream_read.hip",
    "device_checks.hip",
]

ARCH = "gfx950"
CFLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    "-Wall",
    "-Wno-unused-result",
    # Packed fp32 vector instructions stay disabled for every GPU function.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{INCLUDE}",
    f"-I{CSRC}",
]
# Per-source additions.  The decode kernels keep their MFMA accumulators in
# architected VGPRs: the softmax rescale multiplies them on the vector ALU,
# and with accumulators in AGPRs the compiler keeps a VGPR copy of each one,
# refreshed after every MFMA (the rank-64 kernel carried 48 such copies and
# about 50 accumulator moves per 16-token sub-block).
SRC_FLAGS = {
    "lrsa_decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the ROCm toolchain is required to build libprecache.so")


def _compile(src: str, hipcc: str, verbose: bool, checked: bool = False) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ("_checked" if checked else "") + ".o")
    cmd = [hipcc, *CFLAGS, *SRC_FLAGS.get(src, []), *(["-DPRC_DEVICE_CHECKS=1"] if checked else [])]
    if src.endswith(".cpp"):
        cmd += ["-x", "hip"]
    cmd += ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature.
    noise = "is not a recognized feature for this target"
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines() if noise not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{msgs}")
    if verbose and msgs.strip():
        print(msgs, flush=True)
    return obj


def _link(hipcc: str, objs: list[str], path: str, verbose: bool) -> None:
    tmp = path + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}{res.stderr}")
    os.replace(tmp, path)
    if verbose:
        print(f"built {path}", flush=True)


def build(verbose: bool = False, jobs: int | None = None) -> str:
    """Compile every source, link both libraries; returns the release path."""
    hipcc = _hipcc()
    os.makedirs(BUILD_DIR, exist_ok=True)
    units = [(s, False) for s in SOURCES] + [("abi.cpp", True)]
    jobs = jobs or min(len(units), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        objs = list(ex.map(lambda u: _compile(u[0], hipcc, verbose, u[1]), units))
    release, abi_checked = objs[:len(SOURCES)], objs[-1]
    _link(hipcc, release, LIB_PATH, verbose)
    _link(hipcc, [abi_checked if s == "abi.cpp" else o for s, o in zip(SOURCES, release)], CHECKED_LIB_PATH, verbose)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose="-v" in sys.argv)
