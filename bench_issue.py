#!/usr/bin/env python3
"""Issue-rate and co-issue microbenchmark of the attention kernel's per-score
instruction mix on one MI355X (source: bench_issue.hip).

    python bench_issue.py --build    # compile for gfx950 (no GPU needed)
    python bench_issue.py            # run (builds first if needed)

Prints a table: cycles per iteration of each instruction stream with 1, 2
and 4 waves per SIMD, and of each stream in slot 0 of a SIMD while the other
slots run FP4 matrix-core work or the softmax mix.  Every stream is a correct
instruction sequence (no skipped waits, no wrong-output variants).
"""
from __future__ import annotations

import argparse
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(ROOT, "bench_issue.hip")
BIN = os.path.join(ROOT, "_build", "bench_issue")


def build(verbose: bool = False) -> str:
    from paper_2607_24377_amd.build import hipcc

    os.makedirs(os.path.dirname(BIN), exist_ok=True)
    tmp = BIN + f".tmp{os.getpid()}"
    cmd = [hipcc(), "--offload-arch=gfx950", "-O3", "-std=c++17",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        err = "\n".join(l for l in res.stderr.splitlines() if "is not a recognized feature" not in l)
        raise RuntimeError(f"hipcc failed:\n{err}")
    os.replace(tmp, BIN)
    return BIN


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--build", action="store_true", help="only compile")
    args = ap.parse_args()
    if args.build or not os.path.exists(BIN) or os.path.getmtime(BIN) < os.path.getmtime(SRC):
        build(verbose=True)
    if args.build:
        return 0
    return subprocess.run([BIN]).returncode


if __name__ == "__main__":
    sys.exit(main())
