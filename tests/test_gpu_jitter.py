"""Every engine under SDP_FLAG_DEBUG_JITTER: random delays of 0-200 us on the
copy stream, the compute stream and the host thread before each of their
copies, kernels and waits, with the slots poisoned after release where the
mode has slots.  A missing wait between the streams, or between a stream
and the host, would let a kernel read a slot before its copy landed, or a
copy or host thread read a buffer before it was written; the results then
differ from device mode.  Here they must equal device mode bit for bit (and
the oracle, to the parity criteria), for two generator seeds."""
import numpy as np
import pytest

import oracle
from gpu_util import (DevState, HostState, PageableState, check_state, hp_pair, log, need_gpu, rand_inputs,
                      states_equal, to_dev_u16, torch)

pytestmark = pytest.mark.gpu

TILE = 65536
SIZES = [3 * TILE + 5, 1, 70001, 2 * TILE]
R = 3
STEPS = 2


@pytest.fixture(scope="module")
def sdp():
    return need_gpu()


@pytest.fixture(scope="module")
def reference(sdp):
    """Device-mode states after each step (no jitter) and the oracle's."""
    masters, grads = rand_inputs(SIZES, R, STEPS, seed=313)
    hps = [hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t) for t in range(1, STEPS + 1)]
    ctx = sdp.sdp_ctx_create(0, 0, 16, 0)
    dev = DevState(masters, R)
    ref = oracle.State(masters)
    dev_states, ref_states, norms = [], [], []
    try:
        for t in range(STEPS):
            dev.set_grads(grads[t])
            norms.append(sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hps[t][0], 0,
                                               torch.cuda.current_stream().cuda_stream, want_norm=True))
            oracle.step(ref, grads[t], hps[t][1])
            dev_states.append(dev.host())
            ref_states.append(ref.copy())
    finally:
        sdp.sdp_ctx_destroy(ctx)
    return masters, grads, hps, dev_states, ref_states, norms


def jitter_ctx(sdp, monkeypatch, seed, flags, chunk):
    monkeypatch.setenv("SDP_JITTER_SEED", str(seed))
    c = sdp.sdp_ctx_create(0, chunk, 16, flags | sdp.SDP_FLAG_DEBUG_JITTER)
    monkeypatch.delenv("SDP_JITTER_SEED")
    return c


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("mode", ["pinned", "staged", "host_cast"])
def test_streamed_under_jitter_equals_device_mode(sdp, reference, monkeypatch, seed, mode):
    masters, grads, hps, dev_states, ref_states, norms = reference
    flags = sdp.SDP_FLAG_DEBUG_POISON
    if mode == "staged":
        flags |= sdp.SDP_FLAG_STREAM_STAGED
    if mode == "host_cast":
        flags |= sdp.SDP_FLAG_STREAM_HOST_CAST
    log(f"jitter: streamed {mode}, seed {seed}")
    c = jitter_ctx(sdp, monkeypatch, seed, flags, 2 * TILE)
    host = PageableState(sdp, masters, R) if mode == "staged" else HostState(sdp, masters, R)
    try:
        for t in range(STEPS):
            host.set_grads(grads[t])
            n = sdp.sdp_stream_step(c, host.segments(), hps[t][0], TILE)
            assert n == norms[t]
            got = host.host()
            check_state(got, ref_states[t])
            assert states_equal(got, dev_states[t]), f"{mode} under jitter differs from device mode at step {t + 1}"
    finally:
        host.close()
        sdp.sdp_ctx_destroy(c)


@pytest.mark.parametrize("seed", [1, 2])
@pytest.mark.parametrize("fmt", ["f32", "bf16"])
def test_host_route_under_jitter(sdp, reference, monkeypatch, seed, fmt):
    masters, grads, hps, dev_states, ref_states, norms = reference
    log(f"jitter: host route {fmt}, seed {seed}")
    c = jitter_ctx(sdp, monkeypatch, seed, 0, 2 * TILE)
    host = PageableState(sdp, masters, R)
    g = [[torch.zeros(m.size, dtype=torch.int16, device="cuda") for _ in range(R)] for m in masters]
    ref = oracle.State(masters)
    try:
        for t in range(STEPS):
            for s, gs in enumerate(grads[t]):
                for r, x in enumerate(gs):
                    g[s][r].copy_(to_dev_u16(x))
            torch.cuda.synchronize()
            segs = sdp.Segments([(host.p[s].ctypes.data, host.m[s].ctypes.data, host.v[s].ctypes.data,
                                  host.pb[s].ctypes.data, [x.data_ptr() for x in g[s]], host.p[s].size)
                                 for s in range(len(masters))])
            f = sdp.SDP_GBAR_BF16 if fmt == "bf16" else sdp.SDP_GBAR_F32
            n = sdp.sdp_host_update_step(c, segs, hps[t][0], TILE, f)
            assert n == norms[t]
            oracle.step(ref, grads[t], hps[t][1], gbar_bf16=(fmt == "bf16"))
            got = host.host()
            check_state(got, ref)
            if fmt == "f32":
                assert states_equal(got, dev_states[t]), f"route under jitter differs from device mode at step {t + 1}"
    finally:
        host.close()
        sdp.sdp_ctx_destroy(c)


@pytest.mark.parametrize("mode", ["host_cast", "device_cast"])
def test_delivery_under_jitter(sdp, monkeypatch, mode):
    m = sdp.SDP_DELIVER_HOST_CAST if mode == "host_cast" else sdp.SDP_DELIVER_DEVICE_CAST
    c = jitter_ctx(sdp, monkeypatch, 3, 0, 2 * TILE)
    try:
        rng = np.random.default_rng(91)
        for n in (7, 3 * TILE + 5):
            x = (rng.normal(0, 0.02, n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)
            out = torch.full((n,), 0x5555, dtype=torch.int16, device="cuda")
            sdp.sdp_deliver_params(c, x.ctypes.data, out.data_ptr(), n, TILE, m)
            assert np.array_equal(out.cpu().numpy().view(np.uint16), oracle.bf16(x)), n
    finally:
        sdp.sdp_ctx_destroy(c)
