"""Builds libmustafar.so (the gfx950 HIP kernels and their C ABI) in-tree.

    python -m paper_2505_22913_amd.build_lib          # build
    python -m paper_2505_22913_amd.build_lib --asm    # also dump gfx950 assembly

hipcc cross-compiles for gfx950 without a GPU. Packed-FP32 instruction
selection is disabled for every kernel.
"""
from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libmustafar.so")
SOURCES = ["api.hip", "compress.hip", "attention.hip", "attention_mfma.hip", "measure.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: cannot build libmustafar.so")
    return path


def common_flags() -> list[str]:
    return [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-fno-strict-aliasing",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            f"-I{INCLUDE}", f"-I{CSRC}"]


def build(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = [hipcc(), *common_flags(), "-shared", "-o", tmp,
           *[os.path.join(CSRC, s) for s in SOURCES]]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def dump_asm(out_dir: str) -> None:
    """Device assembly of every source, for reading the generated gfx950 code."""
    os.makedirs(out_dir, exist_ok=True)
    for s in SOURCES:
        out = os.path.join(out_dir, s.replace(".hip", f"-{ARCH}.s"))
        cmd = [hipcc(), *common_flags(), "--cuda-device-only", "-S", "-o", out,
               os.path.join(CSRC, s)]
        subprocess.run(cmd, check=True)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--asm", metavar="DIR", help="write gfx950 assembly into DIR")
    ap.add_argument("-v", "--verbose", action="store_true")
    args = ap.parse_args(argv)
    print(build(verbose=args.verbose))
    if args.asm:
        dump_asm(args.asm)
    return 0


if __name__ == "__main__":
    sys.exit(main())
