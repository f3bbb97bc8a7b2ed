"""Runs the CPU test suite against sanitizer builds of the native code
(CPU only; nothing here touches a GPU).

  1. the oracle (oracle/vd_oracle.c, gcc) with AddressSanitizer and
     UndefinedBehaviorSanitizer, aborting on the first report: the oracle's
     pins, the bench's host logic and the oracle baseline leg;
  2. the oracle with ThreadSanitizer (its work queue of host threads): the
     oracle's pins;
  3. libvdattn.so with its host code (the C ABI's checks, the workspace layout,
     the launch planning) built with AddressSanitizer and
     UndefinedBehaviorSanitizer by hipcc's host pass (the device code is built
     as usual): the C ABI tests, which call every entry point's host checks.

The sanitizer runtime is preloaded into the Python process that loads the
instrumented library (Python itself is not instrumented; leak checking is off).
Each build goes to a temporary directory.  Exit status: 0 when every run is
clean.  Usage: python oracle/sanitize.py
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "vd_oracle.c")
CSRC = os.path.join(ROOT, "paper_2609_38981_amd", "csrc")


def gcc_runtime(name: str) -> str:
    return subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True,
                          check=True).stdout.strip()


def clang_asan_runtime() -> str:
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("clang's AddressSanitizer runtime is not installed")
    return hits[-1]


def build_oracle(out: str, flags) -> str:
    subprocess.run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
                    "-fno-fast-math", "-std=c11", "-fPIC", "-shared", "-pthread", *flags,
                    ORACLE_SRC, "-o", out, "-lm"], check=True)
    return out


def build_library(out: str) -> str:
    hipcc = "/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else "hipcc"
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-ffp-contract=off",
           "-fno-fast-math", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-fPIC", "-shared",
           # host pass only
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), os.path.join(CSRC, "vd_attn.hip"),
           os.path.join(CSRC, "vd_linear.hip"), "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stderr)
        raise RuntimeError("hipcc failed")
    return out


def run_tests(name: str, env_extra: dict, tests) -> bool:
    env = dict(os.environ)
    env.update(env_extra)
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu", "-p", "no:cacheprovider",
           *tests]
    print("== %s: %s" % (name, " ".join(tests)), flush=True)
    res = subprocess.run(cmd, cwd=ROOT, env=env)
    print("== %s: %s" % (name, "clean" if res.returncode == 0 else "FAILED (%d)" % res.returncode),
          flush=True)
    return res.returncode == 0


def main() -> int:
    ok = True
    with tempfile.TemporaryDirectory() as tmp:
        lib = build_oracle(os.path.join(tmp, "liboracle_asan.so"),
                           ["-fsanitize=address", "-fsanitize=undefined",
                            "-fno-sanitize-recover=all"])
        ok &= run_tests("oracle, ASan + UBSan", {
            "VDO_ORACLE_LIB": lib,
            "LD_PRELOAD": gcc_runtime("libasan.so") + " " + gcc_runtime("libubsan.so"),
            "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
            "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"},
            ["tests/test_oracle.py", "tests/test_bench_cpu.py"])
        lib = build_oracle(os.path.join(tmp, "liboracle_tsan.so"), ["-fsanitize=thread"])
        # torch single-threaded: its OpenMP threads (uninstrumented libgomp,
        # behind the library pins) would be reported as racing with the main
        # thread; the oracle's own worker threads still run on every core
        ok &= run_tests("oracle, TSan", {
            "VDO_ORACLE_LIB": lib,
            "LD_PRELOAD": gcc_runtime("libtsan.so"),
            "OMP_NUM_THREADS": "1",
            "TSAN_OPTIONS": "halt_on_error=1:report_signal_unsafe=0"},
            ["tests/test_oracle.py"])
        lib = build_library(os.path.join(tmp, "libvdattn_asan.so"))
        ok &= run_tests("libvdattn host code, ASan + UBSan", {
            "VDATTN_LIB": lib,
            "LD_PRELOAD": clang_asan_runtime(),
            "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
            "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"},
            ["tests/test_abi_cpu.py"])
    print("sanitizer runs: %s" % ("all clean" if ok else "FAILED"), flush=True)
    return 0 if ok else 1


if __name__ == "__main__":
    sys.exit(main())
