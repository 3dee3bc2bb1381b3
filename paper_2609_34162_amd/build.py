"""Build libsdp.so for gfx950 with hipcc (in-tree)."""
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "libsdp.so")
SOURCES = [os.path.join(HERE, "csrc", f)
           for f in ("sdp_runtime.hip", "sdp_stream.hip", "sdp_host_route.hip", "sdp_kernels.hip",
                     "sdp_copy.hip", "sdp_noalloc.hip")]
# host-only lanes, built with the host compiler: no fused multiply-add, so the
# FP64 update rounds every product and sum as written
HOST_SOURCES = [os.path.join(HERE, "csrc", f) for f in ("sdp_host_adamw.cpp", "sdp_schedule.cpp")]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HOSTCXX = os.environ.get("SDP_HOSTCXX", "/opt/rocm/llvm/bin/clang++")
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-ffp-contract=off", "-fno-math-errno", "-Wall", "-fvisibility=hidden"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # no packed FP32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
    # only the C ABI (SDP_API in sdp.h) is exported
    "-fvisibility=hidden",
]


def build(verbose: bool = False) -> str:
    tmp = LIB_PATH + ".tmp"
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc")]
    with tempfile.TemporaryDirectory() as d:
        objs = []
        for src in HOST_SOURCES:
            obj = os.path.join(d, os.path.basename(src) + ".o")
            cmd = [HOSTCXX, *HOST_FLAGS, *inc, "-c", src, "-o", obj]
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.check_call(cmd)
            objs.append(obj)
        cmd = [HIPCC, *FLAGS, *inc, "-o", tmp, *SOURCES, "-x", "none", *objs]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
