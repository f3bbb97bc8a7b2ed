"""Builds tests/probes/libvdprobes.so (hipcc, gfx950), the instruction probes
that tests/test_gpu_hw_facts.py runs: test infrastructure, not part of the
attention library.  Same compiler flags as the library."""
from __future__ import annotations

import os
import subprocess
import sys

from paper_2609_38981_amd import build as lib_build

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "vd_probes.hip")
LIB = os.path.join(HERE, "libvdprobes.so")


def build(force: bool = True) -> str:
    if not force and os.path.exists(LIB) and os.path.getmtime(LIB) >= os.path.getmtime(SRC):
        return LIB
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [lib_build.hipcc(), *lib_build.HIPCC_FLAGS, SRC, "-o", tmp]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        err = "\n".join(ln for ln in res.stderr.splitlines() if "packed-fp32-ops" not in ln)
        print(err, file=sys.stderr)
        raise RuntimeError("hipcc failed (%d): %s" % (res.returncode, " ".join(cmd)))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
