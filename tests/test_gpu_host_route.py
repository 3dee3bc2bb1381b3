"""GPU parity of the host-update route (sdp_host_update_step): the R rank
gradients in device memory, the states in host memory (pageable or pinned),
the GPU's norm pass and mean-gradient kernel, chunked copies to the host and
the host threads' AdamW, against the oracle -- with the FP32 mean gradient
(the oracle's plain step) and with the mean gradient rounded to BF16 (the
oracle's BF16-gradient variant).  Criteria as in test_gpu_parity.py.
"""
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_util import (DevState, HostState, PageableState, check_norm, check_state, hp_pair, log, need_gpu,
                      rand_inputs, states_equal, to_dev_u16, torch)

pytestmark = pytest.mark.gpu

TILE = 65536


@pytest.fixture(scope="module")
def sdp():
    return need_gpu()


@pytest.fixture(scope="module")
def ctx(sdp):
    c = sdp.sdp_ctx_create(0, 4 * TILE, 16, 0)
    yield c
    sdp.sdp_ctx_destroy(c)


class RouteState:
    """Host states (pageable numpy arrays, or pinned buffers) and the rank
    gradients on the GPU."""

    def __init__(self, sdp, masters, R, pinned=False):
        self.host = HostState(sdp, masters, R) if pinned else PageableState(sdp, masters, R)
        self.g = [[torch.zeros(m.size, dtype=torch.int16, device="cuda") for _ in range(R)] for m in masters]

    def set_grads(self, grads):
        for s, gs in enumerate(grads):
            for r, g in enumerate(gs):
                self.g[s][r].copy_(to_dev_u16(g))
        torch.cuda.synchronize()

    def segments(self, sdp):
        h = self.host
        return sdp.Segments([(h.p[s].ctypes.data, h.m[s].ctypes.data, h.v[s].ctypes.data, h.pb[s].ctypes.data,
                              [g.data_ptr() for g in self.g[s]], h.p[s].size) for s in range(len(h.p))])

    def state(self):
        return self.host.host()

    def close(self):
        self.host.close()


def fmt_of(sdp, name):
    return sdp.SDP_GBAR_BF16 if name == "bf16" else sdp.SDP_GBAR_F32


@pytest.mark.parametrize("fmt", ["f32", "bf16"])
@pytest.mark.parametrize("chunk_tiles", [1, 3])
@pytest.mark.parametrize("pinned", [False, True])
def test_host_route_matches_oracle(sdp, ctx, fmt, chunk_tiles, pinned):
    sizes = [3 * TILE + 5, 1, 70000, 2 * TILE]
    R = 3
    steps = 3
    masters, grads = rand_inputs(sizes, R, steps, seed=61 + chunk_tiles)
    log(f"host route fmt={fmt} chunk={chunk_tiles} tiles pinned={pinned}")
    st = RouteState(sdp, masters, R, pinned=pinned)
    ref = oracle.State(masters)
    try:
        for t in range(1, steps + 1):
            hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t)
            st.set_grads(grads[t - 1])
            norm = sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, chunk_tiles * TILE, fmt_of(sdp, fmt))
            _, onorm = oracle.step(ref, grads[t - 1], ho, gbar_bf16=(fmt == "bf16"))
            check_norm(norm, onorm)
            assert norm == onorm, "the norm is the exactly rounded one in every mode"
            check_state(st.state(), ref)
    finally:
        st.close()


@pytest.mark.parametrize("fmt", ["f32", "bf16"])
def test_host_route_first_chunk_ramp(sdp, fmt):
    """With 16-tile chunks the pieces grow from one tile by 6/5 (1, 2, 3, 4,
    5 tiles, then the rest of the first segment, 5 tiles and 3 elements, and
    the 5,000-element second segment whole); results still match the oracle,
    and equal those of a chunking too short to ramp (every piece of the
    update is elementwise)."""
    sizes = [20 * TILE + 3, 5000]
    R = 2
    masters, grads = rand_inputs(sizes, R, 2, seed=101)
    c = sdp.sdp_ctx_create(0, 16 * TILE, R, 0)
    a = RouteState(sdp, masters, R)
    b = RouteState(sdp, masters, R)
    ref = oracle.State(masters)
    try:
        for t in (1, 2):
            hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.02, max_grad_norm=0.3, step=t)
            a.set_grads(grads[t - 1])
            b.set_grads(grads[t - 1])
            na = sdp.sdp_host_update_step(c, a.segments(sdp), hs, 16 * TILE, fmt_of(sdp, fmt))
            nb = sdp.sdp_host_update_step(c, b.segments(sdp), hs, TILE, fmt_of(sdp, fmt))
            oracle.step(ref, grads[t - 1], ho, gbar_bf16=(fmt == "bf16"))
            assert na == nb
            check_state(a.state(), ref)
            assert states_equal(a.state(), b.state())
    finally:
        a.close()
        b.close()
        sdp.sdp_ctx_destroy(c)


def test_route_then_delivery_closes_the_loop(sdp, ctx):
    """The paper's per-layer loop on one context: the host route updates the
    host master, then parameter delivery writes its BF16 copy into a device
    window for the next forward pass; the window must equal the route's own
    BF16 params bit for bit, for both delivery modes and both steps."""
    sizes = [3 * TILE + 11, 4097]
    R = 2
    masters, grads = rand_inputs(sizes, R, 2, seed=111)
    st = RouteState(sdp, masters, R)
    try:
        for t in (1, 2):
            hs, _ = hp_pair(sdp, lr=1e-3, weight_decay=0.01, max_grad_norm=0.5, step=t)
            st.set_grads(grads[t - 1])
            sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, 2 * TILE, sdp.SDP_GBAR_BF16)
            for s, n in enumerate(sizes):
                for mode in (sdp.SDP_DELIVER_HOST_CAST, sdp.SDP_DELIVER_DEVICE_CAST):
                    window = torch.full((n,), 0x5555, dtype=torch.int16, device="cuda")
                    sdp.sdp_deliver_params(ctx, st.host.p[s].ctypes.data, window.data_ptr(), n, 2 * TILE, mode)
                    got = window.cpu().numpy().view(np.uint16)
                    assert np.array_equal(got, st.host.pb[s]), (t, s, mode)
    finally:
        st.close()


@pytest.mark.parametrize("mode", ["host_cast", "device_cast"])
@pytest.mark.parametrize("pinned", [False, True])
def test_async_delivery_gates_the_consumer_stream(sdp, ctx, mode, pinned):
    """Event-gated delivery: the call returns with the copies in flight, and
    work that the caller then enqueues on its own stream sees the whole BF16
    window; back-to-back gated deliveries, a blocking one after them and a
    route step after them keep their order and results."""
    m = sdp.SDP_DELIVER_HOST_CAST if mode == "host_cast" else sdp.SDP_DELIVER_DEVICE_CAST
    sizes = [5 * TILE + 13, 3 * TILE]
    R = 2
    masters, grads = rand_inputs(sizes, R, 1, seed=121)
    st = RouteState(sdp, masters, R, pinned=pinned)
    consumer = torch.cuda.Stream()
    try:
        log(f"gated delivery mode={mode} pinned={pinned}")
        wins = [torch.full((n,), 0x5555, dtype=torch.int16, device="cuda") for n in sizes]
        outs = [torch.empty_like(w) for w in wins]
        torch.cuda.synchronize()
        for s, n in enumerate(sizes):
            sdp.sdp_deliver_params_async(ctx, st.host.p[s].ctypes.data, wins[s].data_ptr(), n, TILE, m,
                                         consumer_stream=consumer.cuda_stream)
        with torch.cuda.stream(consumer):
            for w, o in zip(wins, outs):
                o.copy_(w)
        consumer.synchronize()
        for s in range(len(sizes)):
            want = oracle.bf16(st.host.p[s])
            assert np.array_equal(outs[s].cpu().numpy().view(np.uint16), want), s
        # a route step after a gated delivery; then the loop closes with a
        # gated delivery of the updated master and a blocking one beside it
        hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.01, max_grad_norm=0.5, step=1)
        ref = oracle.State(masters)
        sdp.sdp_deliver_params_async(ctx, st.host.p[0].ctypes.data, wins[0].data_ptr(), sizes[0], TILE, m,
                                     consumer_stream=consumer.cuda_stream)
        st.set_grads(grads[0])
        sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, 2 * TILE, sdp.SDP_GBAR_F32)
        oracle.step(ref, grads[0], ho)
        check_state(st.state(), ref)
        sdp.sdp_deliver_params_async(ctx, st.host.p[0].ctypes.data, wins[0].data_ptr(), sizes[0], TILE, m,
                                     consumer_stream=consumer.cuda_stream)
        sdp.sdp_deliver_params(ctx, st.host.p[1].ctypes.data, wins[1].data_ptr(), sizes[1], TILE, m)
        with torch.cuda.stream(consumer):
            outs[0].copy_(wins[0])
        consumer.synchronize()
        assert np.array_equal(outs[0].cpu().numpy().view(np.uint16), st.host.pb[0])
        assert np.array_equal(wins[1].cpu().numpy().view(np.uint16), st.host.pb[1])
    finally:
        torch.cuda.synchronize()
        st.close()


@pytest.mark.parametrize("R", [1, 2, 4, 8, 16])
def test_host_route_ranks_against_device_mode(sdp, ctx, R):
    """FP32 route and device mode: same norm bits, both within the criteria
    of the oracle."""
    sizes = [2 * TILE + 17]
    masters, grads = rand_inputs(sizes, R, 2, seed=70 + R)
    st = RouteState(sdp, masters, R)
    dev = DevState(masters, R)
    ref = oracle.State(masters)
    try:
        for t in (1, 2):
            hs, ho = hp_pair(sdp, lr=2e-3, weight_decay=0.01, max_grad_norm=0.1, step=t)
            st.set_grads(grads[t - 1])
            dev.set_grads(grads[t - 1])
            hn = sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, TILE, sdp.SDP_GBAR_F32)
            dn = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hs, 0, torch.cuda.current_stream().cuda_stream,
                                       want_norm=True)
            torch.cuda.synchronize()
            oracle.step(ref, grads[t - 1], ho)
            assert hn == dn
            check_state(st.state(), ref)
            check_state(dev.host(), ref)
    finally:
        st.close()


def test_host_route_threads_and_simd_give_same_bits(sdp, ctx):
    sizes = [3 * TILE + 3, 999]
    R = 4
    masters, grads = rand_inputs(sizes, R, 1, seed=81)
    hs = sdp.make_params(lr=1e-3, weight_decay=0.1, max_grad_norm=0.5, step=1)
    outs = []
    saved = sdp.sdp_ctx_host_threads(ctx)
    try:
        for threads, simd in ((1, None), (5, None), (16, None), (3, "0")):
            sdp.sdp_ctx_set_host_threads(ctx, threads)
            assert sdp.sdp_ctx_host_threads(ctx) == threads
            if simd is not None:
                os.environ["SDP_HOST_SIMD"] = simd
            st = RouteState(sdp, masters, R)
            try:
                st.set_grads(grads[0])
                sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, 2 * TILE, sdp.SDP_GBAR_BF16)
                outs.append(st.state())
            finally:
                st.close()
                os.environ.pop("SDP_HOST_SIMD", None)
    finally:
        sdp.sdp_ctx_set_host_threads(ctx, saved)
    # worker threads kept on fixed CPUs
    pinned = sdp.sdp_ctx_create(0, 4 * TILE, R, sdp.SDP_FLAG_HOST_PIN_THREADS)
    st = RouteState(sdp, masters, R)
    try:
        st.set_grads(grads[0])
        sdp.sdp_host_update_step(pinned, st.segments(sdp), hs, 2 * TILE, sdp.SDP_GBAR_BF16)
        outs.append(st.state())
    finally:
        st.close()
        sdp.sdp_ctx_destroy(pinned)
    for o in outs[1:]:
        assert states_equal(outs[0], o)


@pytest.mark.parametrize("bad", [np.nan, np.inf])
def test_host_route_nonfinite_leaves_states_unchanged(sdp, ctx, bad):
    sizes = [TILE + 9]
    R = 2
    masters, grads = rand_inputs(sizes, R, 1, seed=91)
    g = [[x.copy() for x in grads[0][0]]]
    g[0][1][4321] = synth.to_bf16_bits(np.array([bad], np.float32))[0]
    st = RouteState(sdp, masters, R)
    try:
        st.host.pb[0][:] = 7
        st.set_grads(g)
        before = st.state()
        with pytest.raises(sdp.SdpNonFinite) as e:
            sdp.sdp_host_update_step(ctx, st.segments(sdp), sdp.make_params(step=1), TILE, sdp.SDP_GBAR_F32)
        assert not np.isfinite(e.value.norm)
        assert states_equal(before, st.state())
    finally:
        st.close()


def test_host_route_argument_errors(sdp, ctx):
    n, R = 4096, 2
    masters, grads = rand_inputs([n], R, 1, seed=95)
    st = RouteState(sdp, masters, R)
    dev = DevState(masters, R)
    L = sdp._lib
    hs = sdp.make_params(step=1)
    try:
        st.set_grads(grads[0])
        dev.set_grads(grads[0])
        before = st.state()
        good = st.segments(sdp)

        def call(segs=good, chunk=TILE, fmt=sdp.SDP_GBAR_F32, c=ctx):
            return L.sdp_host_update_step(c, segs.ptr, segs.n, hs, chunk, fmt, None)

        assert call(fmt=5) == sdp.SDP_ERR_INVALID_ARGUMENT
        assert call(chunk=TILE + 1) == sdp.SDP_ERR_INVALID_ARGUMENT
        assert call(chunk=8 * TILE) == sdp.SDP_ERR_CHUNK_TOO_LARGE
        # states in device memory are refused
        assert call(segs=dev.segments(sdp)) == sdp.SDP_ERR_INVALID_ARGUMENT
        assert "device memory" in sdp.sdp_last_error()
        # gradients in host memory are refused
        h = st.host
        host_grads = sdp.Segments([(h.p[0].ctypes.data, h.m[0].ctypes.data, h.v[0].ctypes.data,
                                    h.pb[0].ctypes.data, [g.ctypes.data for g in h.g[0]], n)])
        assert call(segs=host_grads) == sdp.SDP_ERR_NOT_DEVICE_MEMORY
        nostage = sdp.sdp_ctx_create(0, 0, 4, 0)
        try:
            assert call(c=nostage) == sdp.SDP_ERR_CHUNK_TOO_LARGE
        finally:
            sdp.sdp_ctx_destroy(nostage)
        assert states_equal(before, st.state())
        # gated delivery: the same checks as the blocking one, before any work
        window = torch.full((n,), 0x5555, dtype=torch.int16, device="cuda")
        s = torch.cuda.current_stream().cuda_stream
        deliver = L.sdp_deliver_params_async
        assert deliver(ctx, h.p[0].ctypes.data, window.data_ptr(), n, TILE, 7, s) == sdp.SDP_ERR_INVALID_ARGUMENT
        assert deliver(ctx, h.p[0].ctypes.data, window.data_ptr(), n, TILE + 1, 0, s) == sdp.SDP_ERR_INVALID_ARGUMENT
        assert deliver(ctx, h.p[0].ctypes.data, window.data_ptr(), n, 8 * TILE, 0, s) == sdp.SDP_ERR_CHUNK_TOO_LARGE
        assert deliver(ctx, h.p[0].ctypes.data, window.data_ptr() + 2, n, TILE, 0, s) == sdp.SDP_ERR_ALIGNMENT
        assert deliver(ctx, h.p[0].ctypes.data, h.pb[0].ctypes.data, n, TILE, 0, s) == sdp.SDP_ERR_NOT_DEVICE_MEMORY
        torch.cuda.synchronize()
        assert np.all(window.cpu().numpy().view(np.uint16) == 0x5555)
    finally:
        st.close()


def test_host_route_f32_equals_device_mode_bitwise(sdp, ctx):
    """The host lane evaluates the fused kernel's FP64 expression with the
    same per-step constants and no fused multiply-add on either side, so the
    route with the FP32 mean gradient gives device mode's bits exactly."""
    sizes = [3 * TILE + 5, 70001]
    R = 4
    steps = 3
    masters, grads = rand_inputs(sizes, R, steps, seed=77)
    st = RouteState(sdp, masters, R)
    dev = DevState(masters, R)
    try:
        for t in range(1, steps + 1):
            hs, _ = hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t)
            st.set_grads(grads[t - 1])
            nr = sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, 2 * TILE, sdp.SDP_GBAR_F32)
            dev.set_grads(grads[t - 1])
            nd = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hs, 0, torch.cuda.current_stream().cuda_stream,
                                       want_norm=True)
            torch.cuda.synchronize()
            assert nr == nd
            assert states_equal(st.state(), dev.host()), f"step {t}: host route differs from device mode"
    finally:
        st.close()
