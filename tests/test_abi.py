"""The C-ABI library loads, exports what include/sdp.h declares, and its
host-only logic (planning, byte accounting, argument checks that fail before
any GPU call) behaves as documented.  No compute call is made."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sdp.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w \*]*?\b(sdp_\w+)\s*\(", text, flags=re.M)))


def header_defines():
    out = {}
    for name, val in re.findall(r"^#define\s+(SDP_\w+)\s+\(?(-?(?:0x)?[0-9a-fA-F]+)u?\)?", open(HEADER).read(), flags=re.M):
        out[name] = int(val, 0)
    return out


@pytest.fixture(scope="module")
def sdp():
    from paper_2609_34162_amd import sdp as mod
    return mod


def test_exports_every_declared_symbol(sdp):
    names = header_functions()
    assert len(names) == 32, names
    lib = ctypes.CDLL(sdp.LIB_PATH)
    missing = [n for n in names if not hasattr(lib, n)]
    assert not missing, missing
    # and the binding wraps every one of them under the same name
    unwrapped = [n for n in names if not hasattr(sdp, n)]
    assert not unwrapped, unwrapped


def test_binding_constants_match_header(sdp):
    d = header_defines()
    for name, val in d.items():
        if name in ("SDP_H",):
            continue
        assert getattr(sdp, name) == val, name


def test_status_strings(sdp):
    for name in ("SDP_OK", "SDP_ERR_INVALID_ARGUMENT", "SDP_ERR_ALIGNMENT", "SDP_ERR_NOT_DEVICE_MEMORY",
                 "SDP_ERR_NOT_PINNED", "SDP_ERR_CHUNK_TOO_LARGE", "SDP_ERR_OUT_OF_MEMORY",
                 "SDP_ERR_HIP", "SDP_ERR_NONFINITE"):
        assert sdp.sdp_status_string(getattr(sdp, name)) == name
    assert sdp.sdp_status_string(-99) == "SDP_ERR_UNKNOWN"


def test_plan_matches_workload_shapes(sdp):
    from synth import configs
    want = {0: (1, 16), 1: (12, 2945), 2: (10, 5041), 3: (448, 225380), 4: (14, 13393)}
    for w in configs.WORKLOADS:
        got = sdp.sdp_plan([s.numel for s in w.segments], w.chunk)
        assert got == want[w.cid], (w.name, got)
    assert sdp.sdp_plan([1, 65536, 65537], 65536) == (1 + 1 + 2, 1 + 1 + 2)


def test_plan_rejects_bad_chunks(sdp):
    for chunk in (0, -65536, 1000, 65536 + 1):
        with pytest.raises(sdp.SdpError) as e:
            sdp.sdp_plan([10], chunk)
        assert e.value.status == sdp.SDP_ERR_INVALID_ARGUMENT
    with pytest.raises(sdp.SdpError):
        sdp.sdp_plan([0], 65536)


def test_bytes_per_element(sdp):
    # device mode: norm pass reads 2R; update reads 2R + 12 and writes 14
    for R in (1, 2, 3, 4):
        assert sdp.sdp_bytes_per_elem(False, R) == (26.0 + 4 * R, 0.0)
    # above R = 4 the mean gradient is stored (4 B written, 4 B read back)
    for R in (5, 8, 16):
        assert sdp.sdp_bytes_per_elem(False, R) == (34.0 + 2 * R, 0.0)
    assert sdp.sdp_bytes_per_elem(False, 8, sdp.SDP_FLAG_DEVICE_GBAR_NEVER) == (58.0, 0.0)
    assert sdp.sdp_bytes_per_elem(False, 2, sdp.SDP_FLAG_DEVICE_GBAR_ALWAYS) == (38.0, 0.0)
    # streamed: each gradient crosses once, states in and out
    assert sdp.sdp_bytes_per_elem(True, 4) == (20.0, 14.0)
    assert sdp.sdp_bytes_per_elem(True, 4, sdp.SDP_FLAG_STREAM_GBAR_NEVER) == (28.0, 14.0)
    # BF16 parameters rounded on the host: master, m and v come back, 12 B
    assert sdp.sdp_bytes_per_elem(True, 4, sdp.SDP_FLAG_STREAM_HOST_CAST) == (20.0, 12.0)
    assert sdp.sdp_bytes_per_elem(True, 2, sdp.SDP_FLAG_STREAM_HOST_CAST | sdp.SDP_FLAG_STREAM_STAGED) == (16.0, 12.0)


def test_training_state_bytes_match_paper_table(sdp):
    """Per parameter, the paper's training-state table lists BF16 weights and
    BF16 gradients (2 B each), an FP32 master (4 B) and two FP32 moments
    (8 B): 16 B.  The library's streamed mode moves exactly that state once
    each way at R = 1 with the mean gradient kept on the GPU: in, the
    gradient and the FP32 master and moments; out, the FP32 master and
    moments and the BF16 weights."""
    import json
    fx = json.load(open(os.path.join(ROOT, "tests", "golden", "training_state_bytes.json")))
    b = fx["bytes_per_param"]
    assert fx["total_bytes_per_param"] == sum(b.values()) == 16
    h2d, d2h = sdp.sdp_bytes_per_elem(True, 1, 0)
    assert h2d == b["gradients_bf16"] + b["master_fp32"] + b["adam_moments_fp32"]
    assert d2h == b["master_fp32"] + b["adam_moments_fp32"] + b["compute_weights_bf16"]
    # and every state byte of the table crosses exactly once in one direction or the other
    assert h2d + d2h - (b["master_fp32"] + b["adam_moments_fp32"]) == fx["total_bytes_per_param"]


def test_null_arguments_fail_before_any_gpu_call(sdp):
    L = sdp._lib
    assert L.sdp_agg_adam_step(None, None, 0, None, 0, None, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_stream_step(None, None, 0, None, 65536, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_grad_norm(None, None, 0, 1, 0, None, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_cast_bf16(None, None, None, 0, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_host_update_step(None, None, 0, None, 65536, 0, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_host_adamw(None, None, None, None, None, None, 0, 0, 1.0, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_ctx_set_host_threads(None, 4) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_probe_host_copy(None, None, None, 16, 1, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_deliver_params(None, None, None, 1, 65536, 0) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_deliver_params_async(None, None, None, 1, 65536, 0, None) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_ctx_create(None, 0, 0, 1, 0) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert "NULL" in sdp.sdp_last_error()
    out = ctypes.c_void_p()
    assert L.sdp_ctx_create(ctypes.byref(out), 0, 0, 0, 0) == sdp.SDP_ERR_INVALID_ARGUMENT  # max_ranks 0
    assert L.sdp_ctx_create(ctypes.byref(out), 0, 1000, 4, 0) == sdp.SDP_ERR_INVALID_ARGUMENT  # chunk
    assert L.sdp_ctx_create(ctypes.byref(out), 0, 0, 4, 3) == sdp.SDP_ERR_INVALID_ARGUMENT  # exclusive flags
    assert L.sdp_ctx_create(ctypes.byref(out), 0, 0, 4, 0x100) == sdp.SDP_ERR_INVALID_ARGUMENT  # unknown flag
    assert "unknown" in sdp.sdp_last_error()
