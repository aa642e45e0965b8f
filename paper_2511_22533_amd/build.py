"""Compile the gfx950 kernels and the C-ABI host library into lib/libf3c.so,
and the torch-free command-line driver lib/f3c_drive linked against it.

Every HIP source is compiled with hipcc for gfx950 only. Packed-FP32 VALU
instructions are disabled and floating-point contraction is off (the scoring and
Euler kernels must round every operation as written). Objects are built in
parallel, then linked into one shared library next to this file.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB_DIR = os.path.join(HERE, "lib")
LIB = os.path.join(LIB_DIR, "libf3c.so")
DRIVER = os.path.join(LIB_DIR, "f3c_drive")
ROOT = os.path.dirname(HERE)

SOURCES = ["k_select.hip", "k_rows.hip", "k_gemm.hip", "k_attn.hip", "k_occupancy.hip", "f3c.cpp"]
DRIVER_SOURCE = "f3c_drive.hip"

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-ffp-contract=off",
    "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I" + os.path.join(ROOT, "include"),
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


# Per-source extra flags. The attention kernel runs its softmax on the MFMA
# accumulators with VALU instructions, so they are kept in VGPRs (no AGPR copies).
EXTRA = {"k_attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _compile(src: str, obj: str) -> None:
    cmd = [hipcc(), *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if out.strip():
        print(out, file=sys.stderr)


def build(verbose: bool = False) -> str:
    obj_dir = os.path.join(LIB_DIR, "obj")
    os.makedirs(obj_dir, exist_ok=True)
    srcs = SOURCES + [DRIVER_SOURCE]
    objs = [os.path.join(obj_dir, s.rsplit(".", 1)[0] + ".o") for s in srcs]
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        list(ex.map(_compile, srcs, objs))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs[:-1]]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout)
    os.replace(tmp, LIB)
    tmp = DRIVER + ".tmp"
    cmd = [hipcc(), "--offload-arch=gfx950", "-o", tmp, objs[-1], "-L" + LIB_DIR, "-lf3c", "-Wl,-rpath,$ORIGIN"]
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("driver link failed:\n" + r.stdout)
    os.replace(tmp, DRIVER)
    if verbose:
        print("built", LIB, "and", DRIVER)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
