"""GPU parity at the full workload sizes, in the launch configuration bench.py
times: one Qwen3-8B layer (192,946,176 params, R = 4, 10 steps) and one
Qwen2.5-72B layer (877,674,496 params, R = 8, 3 steps) in device mode, and one
Qwen3-14B layer (330,311,680 params, R = 4, 5 steps) in streamed mode (pinned
host state; pinned with the BF16 parameters rounded on the host; pageable
host state through the staged mode) and on the host-update route (FP32 mean
gradient, 5 steps; BF16 mean gradient, 3 steps; pageable host states,
gradients in device memory), and one segment
of 2^31 + 4099 elements in device mode and on the host-update route
(sampled points, exact norm).

Every element of every output is compared with the oracle at every step,
teacher-forced (the oracle steps from the GPU's state before the step) and,
where stated, also free-running (the oracle carries its own state from step
one).  Criteria as in test_gpu_parity.py.  The full Qwen3-14B model
(14.8B params, 266 GB of pageable host state) is in test_gpu_full_model.py.
"""
import time

import numpy as np
import pytest

import oracle
import synth
from gpu_util import (DevState, HostState, PageableState, check_bf16, check_f32, check_norm, check_state, log,
                      need_gpu, states_equal, torch)

pytestmark = [pytest.mark.gpu, pytest.mark.big]


@pytest.fixture(scope="module")
def sdp():
    return need_gpu()


class Pinned:
    """Reusable pinned host arrays."""

    def __init__(self, sdp):
        self.sdp = sdp
        self.bufs = []

    def array(self, dtype, n):
        b = self.sdp.HostBuffer(max(16, n * np.dtype(dtype).itemsize))
        self.bufs.append(b)
        return b.view(dtype, n)

    def state(self, sizes):
        st = oracle.State([np.zeros(0, np.float32) for _ in sizes])
        st.master = [self.array(np.float32, n) for n in sizes]
        st.exp_avg = [self.array(np.float32, n) for n in sizes]
        st.exp_avg_sq = [self.array(np.float32, n) for n in sizes]
        st.param_bf16 = [self.array(np.uint16, n) for n in sizes]
        return st

    def close(self):
        """Views keep their buffers alive; dropping the list frees the rest."""
        self.bufs = []


def copy_state(dst: oracle.State, src: oracle.State):
    for a, b in ((dst.master, src.master), (dst.exp_avg, src.exp_avg), (dst.exp_avg_sq, src.exp_avg_sq),
                 (dst.param_bf16, src.param_bf16)):
        for s in range(len(a)):
            np.copyto(a[s], b[s])


def dev_to_host(dst: oracle.State, dev: DevState):
    torch.cuda.synchronize()
    for s in range(len(dev.p)):
        torch.from_numpy(dst.master[s]).copy_(dev.p[s])
        torch.from_numpy(dst.exp_avg[s]).copy_(dev.m[s])
        torch.from_numpy(dst.exp_avg_sq[s]).copy_(dev.v[s])
        torch.from_numpy(dst.param_bf16[s].view(np.int16)).copy_(dev.pb[s])


def gen_grads(w, step, out):
    for s in range(len(w.segments)):
        for r in range(w.ranks):
            synth.grad_bf16(w, s, step, r, out=out[s][r])


def run_device_workload(sdp, cid, free_running):
    w = synth.workload(cid)
    sizes = [s.numel for s in w.segments]
    log(f"full device workload {w.name}: N={w.numel} R={w.ranks} steps={w.steps}")
    t0 = time.time()
    pin = Pinned(sdp)
    try:
        masters = [synth.master(w, s) for s in range(len(sizes))]
        dev = DevState(masters, w.ranks)
        grads = [[pin.array(np.uint16, n) for _ in range(w.ranks)] for n in sizes]
        before, after = pin.state(sizes), pin.state(sizes)
        forced = oracle.State([np.zeros(n, np.float32) for n in sizes])
        ref = oracle.State(masters) if free_running else None
        del masters
        ctx = sdp.sdp_ctx_create(0, 0, w.ranks, 0)
        try:
            for t in range(1, w.steps + 1):
                gen_grads(w, t, grads)
                dev.set_grads(grads)
                dev_to_host(before, dev)
                norm = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), sdp.make_params(**w.hparams(t)), w.chunk,
                                             torch.cuda.current_stream().cuda_stream, want_norm=True)
                dev_to_host(after, dev)
                copy_state(forced, before)
                rc, fnorm = oracle.step(forced, grads, oracle.hparams(**w.hparams(t)))
                assert rc == oracle.ORC_OK
                check_norm(norm, fnorm)
                assert norm > w.max_grad_norm      # these workloads clip every step
                stats = check_state(after, forced)
                if ref is not None:
                    oracle.step(ref, grads, oracle.hparams(**w.hparams(t)))
                    stats_free = check_state(after, ref)
                else:
                    stats_free = None
                log(f"  step {t}: norm {norm:.9g} (oracle {fnorm:.9g}) forced {stats['master0']}"
                    f" free {stats_free['master0'] if stats_free else '-'}  {time.time() - t0:.0f}s")
        finally:
            sdp.sdp_ctx_destroy(ctx)
    finally:
        pin.close()


@pytest.mark.timeout(400)
def test_qwen3_8b_layer_device_full(sdp):
    run_device_workload(sdp, 1, free_running=True)


@pytest.mark.timeout(400)
def test_qwen25_72b_layer_device_full(sdp):
    run_device_workload(sdp, 4, free_running=True)


@pytest.mark.timeout(400)
@pytest.mark.parametrize("mode", ["pinned", "pinned_host_cast", "staged"])
def test_qwen3_14b_layer_streamed_full(sdp, mode):
    """The Qwen3-14B layer streamed: pinned host state; pinned with the BF16
    parameters rounded on the host; pageable host state through the staged
    mode.  Released slots are poisoned, so a missing wait shows."""
    w = synth.workload(2)
    n = w.numel
    log(f"full streamed workload {w.name} ({mode}): N={n} R={w.ranks} chunk={w.chunk} steps={w.steps}")
    t0 = time.time()
    flags = sdp.SDP_FLAG_DEBUG_POISON | {"pinned": 0, "pinned_host_cast": sdp.SDP_FLAG_STREAM_HOST_CAST,
                                         "staged": sdp.SDP_FLAG_STREAM_STAGED}[mode]
    ctx = sdp.sdp_ctx_create(0, w.chunk, w.ranks, flags)  # its pinned buffers before the host state
    master = synth.master(w, 0)
    host = (PageableState if mode == "staged" else HostState)(sdp, [master], w.ranks)
    pin = Pinned(sdp)
    try:
        before = pin.state([n])
        forced = oracle.State([np.zeros(n, np.float32)])
        ref = oracle.State([master])
        del master
        for t in range(1, w.steps + 1):
            gen_grads(w, t, host.g)
            for a, b in ((before.master, host.p), (before.exp_avg, host.m), (before.exp_avg_sq, host.v),
                         (before.param_bf16, host.pb)):
                np.copyto(a[0], b[0])
            norm = sdp.sdp_stream_step(ctx, host.segments(), sdp.make_params(**w.hparams(t)), w.chunk)
            after = oracle.State.__new__(oracle.State)
            after.master, after.exp_avg, after.exp_avg_sq, after.param_bf16 = host.p, host.m, host.v, host.pb
            copy_state(forced, before)
            rc, fnorm = oracle.step(forced, host.g, oracle.hparams(**w.hparams(t)))
            assert rc == oracle.ORC_OK
            check_norm(norm, fnorm)
            stats = check_state(after, forced)
            oracle.step(ref, host.g, oracle.hparams(**w.hparams(t)))
            stats_free = check_state(after, ref)
            log(f"  step {t}: norm {norm:.9g} (oracle {fnorm:.9g}) forced {stats['master0']} "
                f"free {stats_free['master0']}  {time.time() - t0:.0f}s")
    finally:
        sdp.sdp_ctx_destroy(ctx)
        host.close()
        pin.close()


@pytest.mark.timeout(300)
def test_qwen3_14b_layer_device_equals_streamed(sdp):
    """The same Qwen3-14B layer in both modes gives the same bits."""
    w = synth.workload(2)
    n = w.numel
    master = synth.master(w, 0)
    host = HostState(sdp, [master], w.ranks)
    dev = DevState([master], w.ranks)
    ctx = sdp.sdp_ctx_create(0, w.chunk, w.ranks, 0)
    pin = Pinned(sdp)
    try:
        got = pin.state([n])
        for t in (1, 2):
            gen_grads(w, t, host.g)
            dev.set_grads(host.g)
            hs = sdp.make_params(**w.hparams(t))
            dn = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hs, w.chunk, torch.cuda.current_stream().cuda_stream,
                                       want_norm=True)
            sn = sdp.sdp_stream_step(ctx, host.segments(), hs, w.chunk)
            assert dn == sn
            dev_to_host(got, dev)
            hstate = oracle.State.__new__(oracle.State)
            hstate.master, hstate.exp_avg, hstate.exp_avg_sq, hstate.param_bf16 = host.p, host.m, host.v, host.pb
            assert states_equal(got, hstate), f"device and streamed modes differ at step {t}"
            log(f"  step {t}: device == streamed, norm {dn:.9g}")
    finally:
        sdp.sdp_ctx_destroy(ctx)
        host.close()
        pin.close()


@pytest.mark.timeout(400)
def test_qwen3_14b_layer_chunk_sizes_agree(sdp):
    """Chunk invariance at the full layer: streamed mode with chunks of one
    tile, 16M and 64M elements gives the device mode's bits and norm (the
    32M chunking is covered above)."""
    w = synth.workload(2)
    n, R = w.numel, w.ranks
    master = synth.master(w, 0)
    pin = Pinned(sdp)
    try:
        grads = [[pin.array(np.uint16, n) for _ in range(R)]]
        gen_grads(w, 1, grads)
        hs = sdp.make_params(**w.hparams(1))
        dev = DevState([master], R)
        dev.set_grads(grads)
        ctx = sdp.sdp_ctx_create(0, 0, R, 0)
        try:
            dn = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hs, 0, torch.cuda.current_stream().cuda_stream,
                                       want_norm=True)
        finally:
            sdp.sdp_ctx_destroy(ctx)
        got = pin.state([n])
        dev_to_host(got, dev)
        del dev
        torch.cuda.empty_cache()
        for chunk in (65536, 1 << 24, 1 << 26):
            host = HostState(sdp, [master], R)
            ctx = sdp.sdp_ctx_create(0, chunk, R, 0)
            try:
                for r in range(R):
                    np.copyto(host.g[0][r], grads[0][r])
                sn = sdp.sdp_stream_step(ctx, host.segments(), hs, chunk)
                hstate = oracle.State.__new__(oracle.State)
                hstate.master, hstate.exp_avg, hstate.exp_avg_sq, hstate.param_bf16 = host.p, host.m, host.v, host.pb
                assert sn == dn, chunk
                assert states_equal(got, hstate), f"chunk {chunk} differs from device mode"
                log(f"  chunk {chunk}: streamed == device, norm {sn:.9g}")
            finally:
                sdp.sdp_ctx_destroy(ctx)
                host.close()
    finally:
        pin.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("fmt", ["f32", "bf16"])
def test_qwen3_14b_layer_host_route_full(sdp, fmt):
    w = synth.workload(2)
    n, R = w.numel, w.ranks
    steps = w.steps if fmt == "f32" else 3
    bf = fmt == "bf16"
    log(f"full host route {w.name} fmt={fmt}: N={n} R={R} chunk={w.chunk} steps={steps}")
    t0 = time.time()
    master = synth.master(w, 0)
    host = PageableState(sdp, [master], R)
    devg = [torch.empty(n, dtype=torch.int16, device="cuda") for _ in range(R)]
    ctx = sdp.sdp_ctx_create(0, w.chunk, R, 0)
    pin = Pinned(sdp)
    try:
        before = pin.state([n])
        forced = oracle.State([np.zeros(n, np.float32)])
        ref = oracle.State([master])
        del master
        segs = sdp.Segments([(host.p[0].ctypes.data, host.m[0].ctypes.data, host.v[0].ctypes.data,
                              host.pb[0].ctypes.data, [g.data_ptr() for g in devg], n)])
        for t in range(1, steps + 1):
            gen_grads(w, t, host.g)
            for r in range(R):
                devg[r].copy_(torch.from_numpy(host.g[0][r].view(np.int16)))
            torch.cuda.synchronize()
            for a, b in ((before.master, host.p), (before.exp_avg, host.m), (before.exp_avg_sq, host.v),
                         (before.param_bf16, host.pb)):
                np.copyto(a[0], b[0])
            ts = time.time()
            norm = sdp.sdp_host_update_step(ctx, segs, sdp.make_params(**w.hparams(t)), w.chunk,
                                            sdp.SDP_GBAR_BF16 if bf else sdp.SDP_GBAR_F32)
            step_s = time.time() - ts
            after = oracle.State.__new__(oracle.State)
            after.master, after.exp_avg, after.exp_avg_sq, after.param_bf16 = host.p, host.m, host.v, host.pb
            copy_state(forced, before)
            rc, fnorm = oracle.step(forced, host.g, oracle.hparams(**w.hparams(t)), gbar_bf16=bf)
            assert rc == oracle.ORC_OK
            check_norm(norm, fnorm)
            assert norm == fnorm
            stats = check_state(after, forced)
            oracle.step(ref, host.g, oracle.hparams(**w.hparams(t)), gbar_bf16=bf)
            stats_free = check_state(after, ref)
            log(f"  step {t}: route {step_s:.3f} s, norm {norm:.9g} forced {stats['master0']} "
                f"free {stats_free['master0']}  {time.time() - t0:.0f}s")
    finally:
        sdp.sdp_ctx_destroy(ctx)
        host.close()
        pin.close()


@pytest.mark.timeout(900)
def test_segment_beyond_int32_elements(sdp):
    """One segment of 2^31 + 4099 elements (R = 2), in device mode and then on
    the host-update route (BF16 mean gradient): 64-bit indexing in every
    kernel and copy offset.  The norm over the 2^32 + 8198 gradient values
    must equal the oracle's exactly rounded norm bit for bit; about 200,000
    sampled points (random, both ends and both sides of 2^31) are checked
    element by element against the oracle's update of the same points."""
    N, R = (1 << 31) + 4099, 2
    log(f"segment of {N} elements, R = {R}")
    t0 = time.time()
    master = synth.normal_f32(synth.seed(4242, 1), N, 0.02)
    grads = []
    tmp = np.empty(1 << 26, np.float32)
    for r in range(R):
        g = np.empty(N, np.uint16)
        s = synth.seed(4242, 2, r)
        for a in range(0, N, tmp.size):
            b = min(a + tmp.size, N)
            synth.normal_f32(s, b - a, 1e-3, start=a, outlier_p=0.01, outlier_scale=100.0, out=tmp[:b - a])
            synth.to_bf16_bits(tmp[:b - a], out=g[a:b])
        grads.append(g)
    log(f"  inputs generated  {time.time() - t0:.0f}s")
    rng = np.random.default_rng(77)
    idx = np.unique(np.concatenate([rng.integers(0, N, 200000), np.arange(64), np.arange(N - 64, N),
                                    np.arange((1 << 31) - 64, (1 << 31) + 64)])).astype(np.int64)
    g_rows = np.stack([g[idx] for g in grads], axis=1)
    hp_kw = dict(lr=1e-3, weight_decay=0.01, max_grad_norm=1.0, step=1)
    onorm = oracle.grad_norm([grads])
    c = oracle.clip_coef(onorm, hp_kw["max_grad_norm"])
    log(f"  oracle norm {onorm!r}, clip {c!r}  {time.time() - t0:.0f}s")
    zeros = np.zeros(idx.size, np.float32)

    dev = DevState([master], R)
    dev.set_grads([grads])
    ctx = sdp.sdp_ctx_create(0, 1 << 25, R, 0)
    try:
        norm = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), sdp.make_params(**hp_kw), 0,
                                     torch.cuda.current_stream().cuda_stream, want_norm=True)
        torch.cuda.synchronize()
        assert norm == onorm, (norm, onorm)
        it = torch.from_numpy(idx).to("cuda")
        got = [dev.p[0][it].cpu().numpy(), dev.m[0][it].cpu().numpy(), dev.v[0][it].cpu().numpy(),
               dev.pb[0][it].cpu().numpy().view(np.uint16)]
        want = oracle.update_points(master[idx], zeros, zeros, g_rows, c, oracle.hparams(**hp_kw))
        for a, b, name in zip(got[:3], want[:3], ("master", "exp_avg", "exp_avg_sq")):
            check_f32(a, b, f"device {name}")
        check_bf16(got[3], got[0], want[3])
        log(f"  device mode: norm equal, {idx.size} points match  {time.time() - t0:.0f}s")
        del dev.p, dev.m, dev.v, dev.pb
        torch.cuda.empty_cache()

        host_p = master.copy()
        host_m = np.zeros(N, np.float32)
        host_v = np.zeros(N, np.float32)
        host_pb = np.zeros(N, np.uint16)
        segs = sdp.Segments([(host_p.ctypes.data, host_m.ctypes.data, host_v.ctypes.data, host_pb.ctypes.data,
                              [g.data_ptr() for g in dev.g[0]], N)])
        rnorm = sdp.sdp_host_update_step(ctx, segs, sdp.make_params(**hp_kw), 1 << 25, sdp.SDP_GBAR_BF16)
        assert rnorm == onorm
        want = oracle.update_points(master[idx], zeros, zeros, g_rows, c, oracle.hparams(**hp_kw), gbar_bf16=True)
        for a, b, name in zip((host_p[idx], host_m[idx], host_v[idx]), want[:3],
                              ("master", "exp_avg", "exp_avg_sq")):
            check_f32(a, b, f"host route {name}")
        check_bf16(host_pb[idx], host_p[idx], want[3])
        log(f"  host route: norm equal, {idx.size} points match  {time.time() - t0:.0f}s")
    finally:
        sdp.sdp_ctx_destroy(ctx)
