"""Build the HIP libraries for gfx950 with hipcc, in-tree: libtas.so, and
libtas_check.so, the same entry points with every instance's state verified
after each iteration (TAS_CHECK_INVARIANTS)."""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libtas.so")
CHECK_LIB = os.path.join(PKG, "libtas_check.so")
SOURCES = ["tas_abi.hip", "tas_sim.hip", "tas_pctl.hip", "tas_order.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _command(out: str, defines: list[str]) -> list[str]:
    srcs = [os.path.join(CSRC, s) for s in SOURCES]
    return [HIPCC, "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            # every floating-point step of the adaptive gamma is one rounded
            # IEEE operation, as in its definition: no fused multiply-add
            "-ffp-contract=off",
            "-Wall", "-Wno-unused-function",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC] + defines + ["-o", out] + srcs


def build(verbose: bool = False) -> str:
    """Compile every HIP source into libtas.so and libtas_check.so (always
    recompiles; the two builds run side by side). Returns libtas.so's path."""
    jobs = [(LIB, []), (CHECK_LIB, ["-DTAS_CHECK_INVARIANTS=1"])]
    procs = []
    for out, defines in jobs:
        cmd = _command(out + ".tmp", defines)
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((out, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                            text=True)))
    failed = False
    for out, p in procs:
        log, _ = p.communicate()
        if p.returncode != 0:
            sys.stderr.write(log)
            failed = True
        else:
            os.replace(out + ".tmp", out)
    if failed:
        raise RuntimeError("hipcc failed")
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
