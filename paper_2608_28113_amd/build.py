"""Builds libhscale.so (gfx950) in-tree with hipcc, and beside it
libhscale_probes.so, the benchmark's measurement probes (no part of the
hscale C ABI).

Flags that fix the arithmetic: -ffp-contract=off (no implicit FMA),
-fhip-fp32-correctly-rounded-divide-sqrt (IEEE division), and packed-FP32
instructions disabled (-packed-fp32-ops).
"""
from __future__ import annotations

import os
import subprocess
import sys
from pathlib import Path

PKG = Path(__file__).resolve().parent
ROOT = PKG.parent
CSRC = PKG / "csrc"
SOURCES = [CSRC / "hdiag.hip", CSRC / "search.hip", CSRC / "diag.hip"]  # share csrc/common.h
INCLUDE = ROOT / "include"
LIB = PKG / "libhscale.so"
PROBE_SOURCES = [CSRC / "probes.hip"]
PROBE_LIB = PKG / "libhscale_probes.so"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wextra", "-Werror=return-type",
]


def _hipcc(sources, out: Path, verbose: bool) -> Path:
    tmp = out.with_suffix(".so.tmp%d" % os.getpid())
    cmd = [HIPCC, *FLAGS, "-I", str(INCLUDE), "-I", str(CSRC), "-o", str(tmp), *map(str, sources)]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass warns that it does not know the packed-fp32 feature.
    err = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + err)
    if err and verbose:
        print(err, file=sys.stderr)
    os.replace(tmp, out)
    return out


def build(verbose: bool = False) -> Path:
    _hipcc(PROBE_SOURCES, PROBE_LIB, verbose)
    return _hipcc(SOURCES, LIB, verbose)


if __name__ == "__main__":
    print(build(verbose=True))
