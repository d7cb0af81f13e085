"""Compile the HIP library for gfx950, in-tree.

Produces ``libresbm.so`` (bf16 activations) and ``libresbm_f32.so`` (the fp32
validation build) next to this file.  Run ``python -m paper_2604_11947_amd.build``.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "resbm_kernels.hip")
SRC_MATRIX = os.path.join(PKG, "csrc", "resbm_matrix.hip")
SRC_TWO = os.path.join(PKG, "csrc", "resbm_two.hip")
DEPS = [SRC, SRC_MATRIX, SRC_TWO, os.path.join(PKG, "csrc", "resbm_buffer.hpp"), os.path.join(PKG, "csrc", "resbm_host.hpp"), os.path.join(PKG, "csrc", "resbm_mfma.hpp"), os.path.join(PKG, "csrc", "resbm_plan.hpp"),
        os.path.join(ROOT, "include", "resbm.h")]

LIBS = {"bf16": "libresbm.so", "f32": "libresbm_f32.so"}


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the HIP library)")


def command(variant: str, out: str) -> list[str]:
    cmd = [hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
           # packed fp32 VALU ops stay disabled in every HIP build of this library
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-o", out, SRC, SRC_MATRIX, SRC_TWO]
    if variant == "f32":
        cmd.insert(1, "-DRESBM_IO_F32_BUILD=1")
    return cmd


def lib_path(variant: str = "bf16") -> str:
    return os.path.join(PKG, LIBS[variant])


def build_all(verbose: bool = False) -> list[str]:
    """Compile both variants (in parallel); raises on any compiler error."""
    procs = []
    for variant, name in LIBS.items():
        out = os.path.join(PKG, name)
        tmp = out + ".tmp"
        cmd = command(variant, tmp)
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((out, tmp, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    built = []
    errors = []
    for out, tmp, p in procs:
        log, _ = p.communicate()
        text = log.decode(errors="replace")
        # hipcc's host pass does not know the packed-fp32 feature and says so; harmless
        text = "\n".join(line for line in text.splitlines() if "packed-fp32-ops" not in line)
        if p.returncode != 0:
            errors.append(f"{os.path.basename(out)}:\n{text}")
            continue
        if verbose and text.strip():
            print(text)
        os.replace(tmp, out)
        built.append(out)
    if errors:
        raise RuntimeError("HIP build failed:\n" + "\n".join(errors))
    return built


def up_to_date(variant: str = "bf16") -> bool:
    out = lib_path(variant)
    if not os.path.exists(out):
        return False
    t = os.path.getmtime(out)
    return all(os.path.getmtime(d) <= t for d in DEPS)


if __name__ == "__main__":
    for path in build_all(verbose="-v" in sys.argv):
        print("built", path)
