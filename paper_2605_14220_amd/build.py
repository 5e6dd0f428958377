"""Build libtim.so (the C-ABI library) for gfx950 with hipcc, in-tree.

    python -m paper_2605_14220_amd.build            # build
    python -m paper_2605_14220_amd.build --asm DIR  # also keep the device assembly in DIR
"""

from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libtim.so")
SOURCES = ["lmhead.hip", "lmgrad.hip", "rmsnorm.hip", "mismatch.hip", "seqstats.hip", "ppo.hip", "tim_api.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    # Every floating-point operation is written out explicitly (fmaf where a
    # fused multiply-add is meant); the compiler may not contract a * b + c.
    "-ffp-contract=off",
    # Keep the compiler from forming packed fp32 arithmetic.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-function",
]


def build(asm_dir: str | None = None, verbose: bool = False, defines=(), out: str = LIB) -> str:
    """Compile the library (`defines`: extra NAME=VALUE preprocessor definitions passed to hipcc)."""
    if shutil.which(HIPCC) is None and not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *[f"-D{x}" for x in defines], "-I", INCLUDE, "-I", CSRC,
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", tmp]
    cwd = None
    if asm_dir:
        os.makedirs(asm_dir, exist_ok=True)
        cmd.insert(1, "-save-temps")
        cwd = asm_dir
    if verbose:
        print(" ".join(cmd))
    r = subprocess.run(cmd, cwd=cwd, capture_output=True, text=True)
    log = "\n".join(line for line in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in line)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed ({r.returncode}):\n{log}")
    if verbose and log.strip():
        print(log)
    os.replace(tmp, out)
    return out


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--asm", default=None, help="directory for -save-temps output")
    ap.add_argument("-v", "--verbose", action="store_true")
    ap.add_argument("-D", dest="defines", action="append", default=[], help="NAME=VALUE preprocessor definition")
    ap.add_argument("-o", dest="out", default=LIB)
    args = ap.parse_args(argv)
    print(build(args.asm, args.verbose, args.defines, args.out))


if __name__ == "__main__":
    sys.exit(main())
