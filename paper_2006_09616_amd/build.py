"""Build step of the HIP library (hipcc, gfx950)."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, f) for f in ("dtr_sim.cpp", "dtr_log.cpp", "replay.hip", "replay_log.hip")]
OUT = os.path.join(HERE, "libdtrsim.so")
# the same sources with the in-kernel cycle timers (profile.py); never the product
OUT_PROFILE = os.path.join(HERE, "libdtrsim_prof.so")
ARCH = "gfx950"

FLAGS = ["-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
         # no packed FP32 instructions anywhere in the device code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = False, profile: bool = False) -> str:
    out = OUT_PROFILE if profile else OUT
    tmp = out + ".tmp"
    cmd = ["hipcc", *FLAGS, *(["-DDTR_PROFILE"] if profile else []), "-o", tmp, *SOURCES]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = [l for l in res.stderr.splitlines() if "packed-fp32-ops" not in l and l.strip()]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(noise))
    if verbose and noise:
        print("\n".join(noise), file=sys.stderr)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
