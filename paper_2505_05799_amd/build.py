"""Build libmxmoe.so (HIP for gfx950) in-tree.

    python -m paper_2505_05799_amd.build [--jobs N]

Every call recompiles all sources: this is the "does it build" check as well as
the build.  Objects go to ``_build/`` at the repository root, the library next
to this file.
"""

from __future__ import annotations

import argparse
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libmxmoe.so")

ARCH = "gfx950"
HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 VALU forms stay off (correctness on this hardware generation)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fvisibility=hidden", "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
]


def _hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: libmxmoe.so needs ROCm's hipcc")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(jobs: int | None = None, verbose: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    srcs = sources()
    objs = [os.path.join(BUILD, os.path.basename(s)[:-4] + ".o") for s in srcs]
    jobs = jobs or min(len(srcs), os.cpu_count() or 1, 16)

    def compile_one(so):
        s, o = so
        # the Group-GEMM translation units report their register use
        extra = ["-Rpass-analysis=kernel-resource-usage"] if os.path.basename(s).startswith("gg_") else []
        return _run([hipcc, *HIPCC_FLAGS, *extra, "-c", s, "-o", o])

    with ThreadPoolExecutor(jobs) as ex:
        logs = list(ex.map(compile_one, zip(srcs, objs)))
    # A persistent Group-GEMM kernel that spills VGPRs runs far slower than its
    # register budget allows: say so loudly (the build still succeeds).
    for s, l in zip(srcs, logs):
        for line in l.splitlines():
            if "VGPRs Spill:" in line:
                n = int(line.split("VGPRs Spill:")[1].split()[0])
                if n > 0:
                    print(f"warning: {os.path.basename(s)} spills {n} VGPRs", file=sys.stderr)
    logs = ["\n".join(x for x in l.splitlines() if "remark:" not in x and "-Rpass-analysis" not in x) for l in logs]
    tmp = LIB + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    os.replace(tmp, LIB)
    if verbose:
        for l in logs:
            if l.strip():
                print(l)
    return LIB


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("--jobs", type=int, default=None)
    ap.add_argument("-v", "--verbose", action="store_true")
    args = ap.parse_args()
    print(build(args.jobs, args.verbose))
    sys.exit(0)
