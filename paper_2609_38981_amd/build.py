"""Builds libvdattn.so (HIP, gfx950: paged attention and the linear layer)
in-tree with hipcc."""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "csrc", "vd_attn.hip")
SRC_LINEAR = os.path.join(HERE, "csrc", "vd_linear.hip")
DEPS = [SRC, SRC_LINEAR, os.path.join(HERE, "csrc", "vd_cas.hpp"), os.path.join(HERE, "csrc", "vd_hw.hpp"),
        os.path.join(ROOT, "include", "vdattn.h")]
LIB = os.path.join(HERE, "libvdattn.so")

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    # value-relevant: no implicit multiply-add contraction, no fast math
    "-ffp-contract=off",
    "-fno-fast-math",
    # never emit packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fPIC",
    "-shared",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def build(force: bool = True, verbose: bool = False) -> str:
    if not force and os.path.exists(LIB) and all(
            os.path.getmtime(LIB) >= os.path.getmtime(d) for d in DEPS):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), *HIPCC_FLAGS, "-I", os.path.join(ROOT, "include"), SRC, SRC_LINEAR, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if verbose or res.returncode != 0:
        # hipcc's host pass reports the device-only feature flag as unknown
        err = "\n".join(ln for ln in res.stderr.splitlines() if "packed-fp32-ops" not in ln)
        if err.strip():
            print(err, file=sys.stderr)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d): %s" % (res.returncode, " ".join(cmd)))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(force=True, verbose=True))
