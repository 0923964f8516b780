"""Build libstreamkl.so (the C-ABI library and its gfx950 kernels) in-tree.

Every translation unit under csrc/ is compiled by hipcc for gfx950 in
parallel, then linked into paper_2606_20005_amd/libstreamkl.so. Packed FP32
instructions are disabled for all device code.

    python -m paper_2606_20005_amd.build [-j N] [-v]
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "obj")
LIB = os.path.join(PKG, "libstreamkl.so")
# benchmark-only kernels (measured MFMA peak), kept out of the library's ABI
BENCH_SRC = os.path.join(CSRC, "bench")
BENCH_LIB = os.path.join(PKG, "libstreamkl_bench.so")
ARCH = "gfx950"

CFLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unknown-pragmas",
    f"-I{INCLUDE}", f"-I{CSRC}",
]


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found: the gfx950 library cannot be built")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host pass warns that it does not know the packed-fp32 feature: harmless
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l and l.strip() != "1 warning generated.")
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


def build(jobs: int | None = None, verbose: bool = False) -> str:
    """Compile every csrc/*.hip for gfx950 and link libstreamkl.so (and the benchmark kernels under
    csrc/bench/ into libstreamkl_bench.so); returns the library's path."""
    cc = hipcc()
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    bench_srcs = sorted(glob.glob(os.path.join(BENCH_SRC, "*.hip")))
    if not srcs:
        raise RuntimeError(f"no sources under {CSRC}")
    allsrc = srcs + bench_srcs
    objs = [os.path.join(OBJDIR, ("bench_" if s in bench_srcs else "") + os.path.basename(s)[:-4] + ".o")
            for s in allsrc]
    jobs = jobs or min(len(allsrc), max(1, min(16, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        futs = [ex.submit(_run, [cc, *CFLAGS, "-c", s, "-o", o], verbose) for s, o in zip(allsrc, objs)]
        for f in futs:
            f.result()
    for lib, part in ((LIB, objs[:len(srcs)]), (BENCH_LIB, objs[len(srcs):])):
        if not part:
            continue
        tmp = lib + ".tmp"
        _run([cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *part, "-o", tmp], verbose)
        os.replace(tmp, lib)
    return LIB


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("-j", "--jobs", type=int, default=None)
    ap.add_argument("-v", "--verbose", action="store_true")
    a = ap.parse_args(argv)
    print(build(a.jobs, a.verbose))


if __name__ == "__main__":
    sys.exit(main())
