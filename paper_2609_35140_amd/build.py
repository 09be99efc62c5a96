"""Build libuattn.so (gfx950) in-tree with hipcc.

    python -m paper_2609_35140_amd.build            # build the library
    python -m paper_2609_35140_amd.build --resource-usage   # also print VGPR/LDS/spill figures

Flags that matter for the numerics:
  -ffp-contract=off   no compiler-chosen fused multiply-adds (the kernels
                      spell out every fma they use), so the two attention
                      paths cannot differ by a contraction;
  -Xclang -target-feature -Xclang -packed-fp32-ops
                      no packed fp32 instructions;
  no fast-math, fp32 denormals kept (the default mode for these kernels).
"""
from __future__ import annotations

import argparse
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libuattn.so")

ARCH = "gfx950"
COMMON_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-ffp-contract=off",
    "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libuattn)")


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def build(resource_usage: bool = False, out: str = LIB, verbose: bool = False, defines=()) -> str:
    cmd = [hipcc(), *COMMON_FLAGS, *[f"-D{d}" for d in defines], "-shared", f"-I{INCLUDE}", f"-I{CSRC}", *sources(),
           "-o", out + ".tmp"]
    if resource_usage:
        cmd.insert(1, "-Rpass-analysis=kernel-resource-usage")
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with code {res.returncode}")
    if resource_usage:
        lines = [ln for ln in res.stderr.splitlines() if "remark" in ln or "Function Name" in ln or ":" in ln]
        sys.stdout.write("\n".join(lines) + "\n")
    os.replace(out + ".tmp", out)
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--resource-usage", action="store_true")
    ap.add_argument("-v", "--verbose", action="store_true")
    args = ap.parse_args(argv)
    path = build(resource_usage=args.resource_usage, verbose=args.verbose)
    print(path)


if __name__ == "__main__":
    main()
