"""The C ABI from plain C99 (no GPU): include/sdp.h compiles with
-std=c99 -pedantic -Werror, a C program links libsdp.so and runs the
host-only entry points, and the struct layouts it prints match the ctypes
binding's."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def sdp():
    from paper_2609_34162_amd import sdp as mod
    return mod


def test_c_program_uses_the_abi(sdp, tmp_path):
    exe = tmp_path / "abi_from_c"
    libdir = os.path.dirname(sdp.LIB_PATH)
    # a sanitizer build of the library (SDP_LIB) takes its runtime from the
    # preloaded one, which the program inherits
    extra = ["-Wl,--allow-shlib-undefined"] if os.environ.get("SDP_LIB") else []
    subprocess.check_call(["gcc", "-std=c99", "-pedantic", "-Wall", "-Wextra", "-Werror",
                           "-I", os.path.join(ROOT, "include"), os.path.join(ROOT, "tests", "c", "abi_from_c.c"),
                           "-o", str(exe), "-L", libdir, "-lsdp", f"-Wl,-rpath,{libdir}", *extra])
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    lines = dict((ln.split()[0], [int(x) for x in ln.split()[1:]]) for ln in out.stdout.splitlines()
                 if ln.startswith("sdp_"))
    import ctypes
    assert lines["sdp_adamw_params"] == [ctypes.sizeof(sdp.sdp_adamw_params), sdp.sdp_adamw_params.step.offset]
    assert lines["sdp_segment"] == [ctypes.sizeof(sdp.sdp_segment), sdp.sdp_segment.n_ranks.offset,
                                    sdp.sdp_segment.numel.offset]
    assert lines["sdp_kernel_times"] == [ctypes.sizeof(sdp.sdp_kernel_times),
                                         sdp.sdp_kernel_times.host_adam_elems.offset]
    assert lines["sdp_rates"] == [ctypes.sizeof(sdp.sdp_rates), sdp.sdp_rates.dep_us.offset]
    assert lines["sdp_prediction"] == [ctypes.sizeof(sdp.sdp_prediction), sdp.sdp_prediction.n_chunks.offset]
    assert out.stdout.strip().endswith("ok")
