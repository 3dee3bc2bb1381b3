#!/usr/bin/env python3
"""The CPU test suite with the host C and C++ code built under AddressSanitizer
and UndefinedBehaviorSanitizer: the oracle (oracle/oracle.c), the input
generator (synth/gen.c) and the library's host lanes (the AVX-512 AdamW and
BF16 rounding, sdp_host_adamw.cpp; the step-time model, sdp_schedule.cpp).

All three libraries are built with clang into _build_sanitize/ (the library's
HIP sources unchanged, its two host files instrumented), the clang ASan
runtime is preloaded into Python, and `pytest -m "not gpu"` runs with
ORACLE_LIB, SYNTH_LIB and SDP_LIB pointing at those builds.  Any sanitizer
report aborts the run (halt_on_error).  Leak checking is off: the Python
process and its extensions keep memory until exit by design.

    python3 tests/run_sanitized.py [extra pytest arguments]
"""
import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OUT = os.path.join(ROOT, "_build_sanitize")
LLVM = "/opt/rocm/llvm/bin"
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g", "-O1"]


def run(cmd):
    print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)


def build():
    os.makedirs(OUT, exist_ok=True)
    csrc = os.path.join(ROOT, "paper_2609_34162_amd", "csrc")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", csrc]
    run([f"{LLVM}/clang", *SAN, "-fopenmp", "-fPIC", "-shared", "-std=c11", "-ffp-contract=off",
         "-I", os.path.join(ROOT, "oracle"), "-o", os.path.join(OUT, "liboracle.so"),
         os.path.join(ROOT, "oracle", "oracle.c"), "-lm"])
    run([f"{LLVM}/clang", *SAN, "-fopenmp", "-fPIC", "-shared", "-std=c11",
         "-o", os.path.join(OUT, "libsynth.so"), os.path.join(ROOT, "synth", "gen.c"), "-lm"])
    objs = []
    for f in ("sdp_host_adamw.cpp", "sdp_schedule.cpp"):
        o = os.path.join(OUT, f + ".o")
        run([f"{LLVM}/clang++", *SAN, "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-math-errno",
             "-fvisibility=hidden", *inc, "-c", os.path.join(csrc, f), "-o", o])
        objs.append(o)
    sys.path.insert(0, os.path.join(ROOT, "paper_2609_34162_amd"))
    import build as hipbuild  # noqa: E402  the library's own build script: its HIP sources and flags
    run([HIPCC, *hipbuild.FLAGS, *inc, "-o", os.path.join(OUT, "libsdp.so"), *hipbuild.SOURCES,
         "-x", "none", *objs])


def main():
    build()
    runtime = glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so")[0]
    env = dict(os.environ)
    env.update(LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1:detect_odr_violation=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               ORACLE_LIB=os.path.join(OUT, "liboracle.so"), SYNTH_LIB=os.path.join(OUT, "libsynth.so"),
               SDP_LIB=os.path.join(OUT, "libsdp.so"))
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-m", "not gpu",
           "-p", "no:xdist", "-p", "no:cacheprovider", *sys.argv[1:]]
    print(" ".join(cmd), flush=True)
    return subprocess.call(cmd, env=env, cwd=ROOT)


if __name__ == "__main__":
    sys.exit(main())
