"""Build libzsa.so in-tree with hipcc for gfx950.

Every translation unit is compiled as HIP (-x hip) for gfx950 only, with
packed fp32 instructions disabled, and linked into one shared library next
to this file. ``build()`` always recompiles.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_PATH = os.path.join(HERE, "libzsa.so")

SOURCES = [
    "zsa_api.cpp",
    "zsa_static.cpp",
    "k_norm.hip",
    "k_gemm.hip",
    "k_attn.hip",
    "k_score.hip",
    "k_select.hip",
    "k_gather.hip",
    "k_decode.hip",
    "k_backward.hip",
]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}",
    "-x", "hip",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


# MFMA results in VGPRs rather than the compiler's default choice of
# accumulation registers: the attention, score and backward kernels run
# softmax and scaling VALU work on their accumulators, and in AGPRs every
# such use costs a v_accvgpr read and write (and the register total grows).
# The GEMM file keeps the default: its 128x128-per-wave tiles need the AGPRs.
VGPR_MFMA = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
EXTRA_FLAGS = {
    "k_attn.hip": VGPR_MFMA,
    "k_score.hip": VGPR_MFMA,
    "k_backward.hip": VGPR_MFMA,
    "k_decode.hip": VGPR_MFMA,
}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(
        line for line in (res.stdout + res.stderr).splitlines()
        if "packed-fp32-ops' is not a recognized feature" not in line
    )
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{out}")
    if out.strip():
        sys.stderr.write(out + "\n")
    return obj


def build(verbose: bool = False) -> str:
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(BUILD_DIR, exist_ok=True)
    workers = min(len(SOURCES), max(1, (os.cpu_count() or 2)))
    with concurrent.futures.ThreadPoolExecutor(max_workers=workers) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB_PATH + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"link failed:\n{res.stdout}{res.stderr}")
    os.replace(tmp, LIB_PATH)
    if verbose:
        print(f"built {LIB_PATH}")
    return LIB_PATH


def clean() -> None:
    shutil.rmtree(BUILD_DIR, ignore_errors=True)
    if os.path.exists(LIB_PATH):
        os.remove(LIB_PATH)


if __name__ == "__main__":
    build(verbose=True)
