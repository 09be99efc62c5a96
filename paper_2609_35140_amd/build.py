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
# measured-ceiling microbenchmarks (streaming read, MFMA), a library of their own
CEIL_SRC = os.path.join(PKG, "ceilings", "uattn_ceilings.hip")
CEIL_LIB = os.path.join(PKG, "libuattn_ceilings.so")

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


# Extra flags for single sources.  The backward's dK/dV kernel carries 128 fp32
# accumulators through its loop; by default the compiler parks them in AGPRs
# and copies them to VGPRs and back on every iteration (about 200 moves per
# 128 MFMAs).  Asking for the VGPR form of the MFMAs removes the copies.  Only
# this file: the flag changes the decode kernel's code too.
PER_FILE_FLAGS = {
    "uattn_backward.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form=1"],
}

OBJDIR = os.path.join(PKG, "_build")


def _compile(src: str, defines, resource_usage: bool):
    obj = os.path.join(OBJDIR, os.path.basename(src)[:-4] + ".o")
    cmd = [hipcc(), *COMMON_FLAGS, *PER_FILE_FLAGS.get(os.path.basename(src), []), *[f"-D{d}" for d in defines],
           f"-I{INCLUDE}", f"-I{CSRC}", "-c", src, "-o", obj]
    if resource_usage:
        cmd.insert(1, "-Rpass-analysis=kernel-resource-usage")
    res = subprocess.run(cmd, capture_output=True, text=True)
    return obj, cmd, res


def build(resource_usage: bool = False, out: str = LIB, verbose: bool = False, defines=()) -> str:
    """Compile every source to its own object (in parallel), then link the
    library; then the measured-ceiling library."""
    _build_lib(sources(), out, resource_usage, verbose, defines)
    if out == LIB:
        _build_lib([CEIL_SRC], CEIL_LIB, False, verbose, ())
    return out


def _build_lib(srcs, out, resource_usage, verbose, defines):
    from concurrent.futures import ThreadPoolExecutor
    os.makedirs(OBJDIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        results = list(ex.map(lambda f: _compile(f, defines, resource_usage), srcs))
    for obj, cmd, res in results:
        if verbose:
            print(" ".join(cmd), flush=True)
        if res.returncode != 0:
            sys.stderr.write(res.stdout + res.stderr)
            raise RuntimeError(f"hipcc failed with code {res.returncode} on {os.path.basename(obj)}")
        if resource_usage:
            lines = [ln for ln in res.stderr.splitlines() if "remark" in ln]
            sys.stdout.write("\n".join(lines) + "\n")
    link = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *[obj for obj, _, _ in results], "-o", out + ".tmp"]
    if verbose:
        print(" ".join(link), flush=True)
    res = subprocess.run(link, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"link failed with code {res.returncode}")
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
