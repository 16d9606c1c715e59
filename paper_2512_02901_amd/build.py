"""Build libfairy2i.so (gfx950) in-tree with hipcc.

    python -m paper_2512_02901_amd.build      # or build() from Python

Every source in csrc/ is compiled separately (in parallel) to an object under
_build/ and linked into paper_2512_02901_amd/libfairy2i.so.  Always rebuilds.
"""
from __future__ import annotations

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libfairy2i.so")
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", shutil.which("hipcc") or "/opt/rocm/bin/hipcc")

CXXFLAGS = [
    "-std=c++17", "-O3", "-fPIC", f"--offload-arch={ARCH}",
    # no packed-fp32 (v_pk_*_f32) code generation
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


# per-source extra flags
EXTRA = {
    # keep MFMA accumulators in VGPRs: the decode kernels accumulate across
    # steps and items, and AGPR accumulators cost copies on every step
    "decode.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    # and leave the cooperative kernel's one-lane claim atomics as written (the
    # atomic optimizer would read each result back at once, waiting for every
    # load in flight)
    "decode_f4.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-mllvm", "-amdgpu-atomic-optimizer-strategy=None"],
    # accumulators in VGPRs: the probe loops are then the MFMAs alone
    "probe.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


# host-only sources (the CPU table-lookup kernel): plain C++, no contraction
# of multiply-add pairs, so the double epilogue rounds like the plain formula
HOST_CXX = os.environ.get("CXX", shutil.which("g++") or "g++")
HOST_FLAGS = ["-std=c++17", "-O3", "-fPIC", "-ffp-contract=off", "-pthread", "-Wall",
              "-I", os.path.join(ROOT, "include"), "-I", CSRC]


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith((".hip", ".cpp")))


def object_path(src):
    stem, ext = os.path.splitext(os.path.basename(src))
    return os.path.join(BUILD, stem + (".host.o" if ext == ".cpp" else ".o"))


def _compile(src):
    ext = os.path.splitext(src)[1]
    obj = object_path(src)
    if ext == ".cpp":
        cmd = [HOST_CXX, *HOST_FLAGS, "-c", src, "-o", obj]
    else:
        cmd = [HIPCC, *CXXFLAGS, *EXTRA.get(os.path.basename(src), []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def link(objs):
    tmp = LIB + ".tmp"
    # hipBLASLt: the three real products of the planar complex GEMM
    cmd = [HIPCC, "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-pthread", "-lhipblaslt", "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    link(objs)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
