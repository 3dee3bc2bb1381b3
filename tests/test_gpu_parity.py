"""GPU parity: the HIP path through the C ABI against the oracle, on small
inputs that span several tiles and ragged tails, plus bit-exact invariants.

Criteria (per element, every step): FP32 master / exp_avg / exp_avg_sq within
relative error 1e-5 of the oracle (an oracle zero requires a GPU zero); BF16
params equal to bf16(GPU master) everywhere, equal to bf16(oracle master) on
all but 1e-4 of elements and within 1 BF16 ulp everywhere; gradient norm
within relative 1e-6.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import (DevState, HostState, PageableState, check_norm, check_state, hp_pair, log, need_gpu,
                      rand_inputs, states_equal, torch)

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


@pytest.fixture(scope="module")
def ctx_store(sdp):
    c = sdp.sdp_ctx_create(0, 4 * TILE, 16, sdp.SDP_FLAG_DEVICE_GBAR_ALWAYS)
    yield c
    sdp.sdp_ctx_destroy(c)


@pytest.fixture(scope="module")
def ctx_nostore(sdp):
    c = sdp.sdp_ctx_create(0, 4 * TILE, 16, sdp.SDP_FLAG_DEVICE_GBAR_NEVER | sdp.SDP_FLAG_STREAM_GBAR_NEVER)
    yield c
    sdp.sdp_ctx_destroy(c)


@pytest.fixture(scope="module")
def ctx_poison(sdp):
    c = sdp.sdp_ctx_create(0, 4 * TILE, 16, sdp.SDP_FLAG_DEBUG_POISON)
    yield c
    sdp.sdp_ctx_destroy(c)


def stream():
    return torch.cuda.current_stream().cuda_stream


def dev_step(sdp, ctx, dev, grads, hp, chunk=0, want_norm=True):
    dev.set_grads(grads)
    norm = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hp, chunk, stream(), want_norm=want_norm)
    torch.cuda.synchronize()
    return norm


def test_tiny_workload_free_running_and_teacher_forced(sdp, ctx):
    w = synth.workload(0)
    log(f"workload {w.name}")
    master = synth.master(w, 0)
    dev = DevState([master], w.ranks)
    ref = oracle.State([master])
    for t in range(1, w.steps + 1):
        grads = [[synth.grad_bf16(w, 0, t, r) for r in range(w.ranks)]]
        hs, ho = hp_pair(sdp, **w.hparams(t))
        before = dev.host()
        norm = dev_step(sdp, ctx, dev, grads, hs, chunk=w.chunk)
        rc, onorm = oracle.step(ref, grads, ho)
        assert rc == oracle.ORC_OK
        check_norm(norm, onorm)
        assert norm < w.max_grad_norm  # this workload's clip is a no-op
        got = dev.host()
        check_state(got, ref)                      # free running
        forced = before.copy()
        oracle.step(forced, grads, ho)
        check_state(got, forced)                   # teacher forced


SIZES = [1, 7, 8, 9, 63, 64, 65, 4095, 4097, TILE - 1, TILE, TILE + 1, 3 * TILE + 5]


@pytest.mark.parametrize("R", [1, 2, 3, 4, 5, 8, 16])
@pytest.mark.parametrize("store", [False, True])
def test_sizes_and_ranks(sdp, ctx_store, ctx_nostore, R, store):
    c = ctx_store if store else ctx_nostore
    log(f"sizes/ranks R={R} store={store}")
    for n in SIZES:
        masters, grads = rand_inputs([n], R, 2, seed=1000 + 17 * n + R)
        dev = DevState(masters, R)
        ref = oracle.State(masters)
        for t in (1, 2):
            hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.02, max_grad_norm=0.05, step=t)
            norm = dev_step(sdp, c, dev, grads[t - 1], hs)
            _, onorm = oracle.step(ref, grads[t - 1], ho)
            check_norm(norm, onorm)
            check_state(dev.host(), ref)


def test_multi_segment_with_clipping(sdp, ctx):
    sizes = [2 * TILE + 3, 1, 100000, 8]
    R = 4
    masters, grads = rand_inputs(sizes, R, 3, seed=5)
    dev = DevState(masters, R)
    ref = oracle.State(masters)
    for t in (1, 2, 3):
        hs, ho = hp_pair(sdp, lr=1e-4, weight_decay=0.1, max_grad_norm=0.1, step=t)
        norm = dev_step(sdp, ctx, dev, grads[t - 1], hs)
        _, onorm = oracle.step(ref, grads[t - 1], ho)
        check_norm(norm, onorm)
        assert norm > 0.1  # clipping active
        check_state(dev.host(), ref)


def test_bit_exact_invariants(sdp, ctx, ctx_store, ctx_nostore):
    n = 3 * TILE + 77
    masters, grads = rand_inputs([n], 4, 3, seed=9)
    hs = [sdp.make_params(lr=1e-3, max_grad_norm=0.05, step=t) for t in (1, 2, 3)]

    def run(c, R=4, g=None, params=None, chunk=0, steps=3):
        dev = DevState(masters, R)
        for t in range(steps):
            gg = g[t] if g is not None else grads[t]
            dev_step(sdp, c, dev, gg, (params or hs)[t], chunk=chunk)
        return dev.host()

    base = run(ctx)
    assert states_equal(base, run(ctx)), "repeat run differs"
    assert states_equal(base, run(ctx_store)), "stored g_bar path differs"
    assert states_equal(base, run(ctx_nostore)), "no-store path differs"
    assert states_equal(base, run(ctx, chunk=TILE)), "chunk size changed the result"
    # R identical buffers == R = 1
    one = [[[grads[t][0][0]]] for t in range(3)]
    four = [[[grads[t][0][0]] * 4] for t in range(3)]
    assert states_equal(run(ctx, R=1, g=one), run(ctx, R=4, g=four)), "identical ranks != one rank"
    # clip no-op: a max norm above the norm equals no clipping
    big = [sdp.make_params(lr=1e-3, max_grad_norm=1e6, step=t) for t in (1, 2, 3)]
    off = [sdp.make_params(lr=1e-3, max_grad_norm=0.0, step=t) for t in (1, 2, 3)]
    assert states_equal(run(ctx, params=big), run(ctx, params=off)), "clip no-op differs"
    # resume: 2 steps, copy out, rebuild, step 3
    dev = DevState(masters, 4)
    for t in range(2):
        dev_step(sdp, ctx, dev, grads[t], hs[t])
    h = dev.host()
    dev2 = DevState(h.master, 4, h.exp_avg, h.exp_avg_sq)
    dev_step(sdp, ctx, dev2, grads[2], hs[2])
    assert states_equal(base, dev2.host()), "resume after a state copy differs"
    # lr = 0 leaves the master bit-unchanged
    dev = DevState(masters, 4)
    dev_step(sdp, ctx, dev, grads[0], sdp.make_params(lr=0.0, step=1))
    got = dev.host()
    assert np.array_equal(got.master[0], masters[0])
    assert np.array_equal(got.param_bf16[0], oracle.bf16(masters[0]))


def edge_cases():
    """(name, masters, m, v, grads, hyperparameters) of degenerate inputs."""
    rng = np.random.default_rng(321)
    n = TILE + 37
    R = 2
    out = []
    # all-zero gradients: norm 0, c = 1, decay only, moments scale down
    m0 = (rng.normal(0, 1e-3, n)).astype(np.float32)
    v0 = (rng.random(n) * 1e-6).astype(np.float32)
    z = np.zeros(n, np.uint16)
    out.append(("zero gradients", rng.normal(0, 0.02, n).astype(np.float32), m0, v0, [z, z],
                dict(lr=1e-3, weight_decay=0.1, max_grad_norm=1.0, step=3)))
    # subnormal states and gradients (BF16 has FP32's exponent range)
    tiny = np.float32(1e-40)
    sub = lambda k: (rng.integers(-60, 60, n) * tiny).astype(np.float32)
    gsub = [synth.to_bf16_bits((rng.integers(-60, 60, n) * tiny).astype(np.float32)) for _ in range(R)]
    out.append(("subnormals", sub(0), sub(1), np.abs(sub(2)), gsub,
                dict(lr=1e-3, weight_decay=0.01, eps=1e-45, max_grad_norm=0.0, step=2)))
    # huge gradients near the BF16 maximum: the norm is huge and c tiny
    big = [synth.to_bf16_bits((rng.choice([-1, 1], n) * rng.uniform(1e37, 3e38, n)).astype(np.float32))
           for _ in range(R)]
    out.append(("huge gradients", rng.normal(0, 0.02, n).astype(np.float32), np.zeros(n, np.float32),
                np.zeros(n, np.float32), big, dict(lr=1e-3, weight_decay=0.01, max_grad_norm=1.0, step=1)))
    # masters on BF16 rounding ties, lr = 0 so the master stays put: the BF16
    # output must round every tie to even
    hi = rng.integers(0, 1 << 16, n).astype(np.uint32) & ~np.uint32(0x7f80)   # finite, not NaN/Inf
    hi |= np.uint32(0x3c00)
    ties = ((hi << 16) | 0x8000).view(np.float32)
    g1 = synth.to_bf16_bits(rng.normal(0, 1e-3, n).astype(np.float32))
    out.append(("bf16 ties", ties, np.zeros(n, np.float32), np.zeros(n, np.float32), [g1, g1],
                dict(lr=0.0, weight_decay=0.0, max_grad_norm=1.0, step=1)))
    return out


@pytest.mark.parametrize("case", range(4))
@pytest.mark.parametrize("mode", ["device", "streamed", "route"])
def test_edge_values(sdp, ctx, case, mode):
    name, master, m, v, grads, kw = edge_cases()[case]
    R = len(grads)
    log(f"edge case {name}, {mode}")
    ref = oracle.State([master], [m], [v])
    rc, onorm = oracle.step(ref, [grads], oracle.hparams(**kw))
    assert rc == oracle.ORC_OK
    hs = sdp.make_params(**kw)
    if mode == "device":
        dev = DevState([master], R, [m], [v])
        norm = dev_step(sdp, ctx, dev, [grads], hs)
        got = dev.host()
    elif mode == "streamed":
        host = HostState(sdp, [master], R, [m], [v])
        try:
            host.set_grads([grads])
            norm = sdp.sdp_stream_step(ctx, host.segments(), hs, TILE)
            got = host.host()
        finally:
            host.close()
    else:
        host = PageableState(sdp, [master], R)
        host.m[0][:] = m
        host.v[0][:] = v
        g = [torch.from_numpy(x.view(np.int16)).to("cuda") for x in grads]
        segs = sdp.Segments([(host.p[0].ctypes.data, host.m[0].ctypes.data, host.v[0].ctypes.data,
                              host.pb[0].ctypes.data, [x.data_ptr() for x in g], master.size)])
        norm = sdp.sdp_host_update_step(ctx, segs, hs, TILE, sdp.SDP_GBAR_F32)
        got = host.host()
    assert norm == onorm, (name, norm, onorm)
    check_state(got, ref)
    if name == "bf16 ties":
        assert np.array_equal(got.master[0], master)
        assert np.array_equal(got.param_bf16[0], oracle.bf16(master))


@pytest.mark.parametrize("R", [4, 8])
def test_residency_cap_does_not_change_results(sdp, R, monkeypatch):
    """The residency caps of the fused update (one-wave blocks, at most 10
    per compute unit) and of the norm pass that stores g_bar (at most 3) are
    launch shapes only: uncapped, the default caps and caps of 3 give the
    same bits and norm, also with the capped grid-stride launch of
    SDP_UPDATE_MAX_BLOCKS.  At R = 8 the norm pass stores g_bar."""
    n = 5 * TILE + 13
    masters, grads = rand_inputs([n], R, 2, seed=141 + R)
    outs, norms = [], []
    for per_cu, max_blocks in (("0", None), (None, None), ("3", None), (None, "40")):
        for name, val in (("SDP_UPDATE_BLOCKS_PER_CU", per_cu), ("SDP_NORM_STORE_BLOCKS_PER_CU", per_cu),
                          ("SDP_UPDATE_MAX_BLOCKS", max_blocks)):
            if val is None:
                monkeypatch.delenv(name, raising=False)
            else:
                monkeypatch.setenv(name, val)
        c = sdp.sdp_ctx_create(0, 0, R, 0)  # reads the variables
        try:
            dev = DevState(masters, R)
            got = []
            for t in (1, 2):
                hs, _ = hp_pair(sdp, lr=1e-3, weight_decay=0.02, max_grad_norm=0.05, step=t)
                got.append(dev_step(sdp, c, dev, grads[t - 1], hs))
            outs.append(dev.host())
            norms.append(got)
        finally:
            sdp.sdp_ctx_destroy(c)
    for name in ("SDP_UPDATE_BLOCKS_PER_CU", "SDP_NORM_STORE_BLOCKS_PER_CU", "SDP_UPDATE_MAX_BLOCKS"):
        monkeypatch.delenv(name, raising=False)
    ref = oracle.State(masters)
    for t in (1, 2):
        _, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.02, max_grad_norm=0.05, step=t)
        oracle.step(ref, grads[t - 1], ho)
    check_state(outs[0], ref)
    for o, nm in zip(outs[1:], norms[1:]):
        assert states_equal(outs[0], o)
        assert nm == norms[0]


@pytest.mark.parametrize("R", [4, 8])
def test_update_pattern_probe(sdp, ctx, R):
    """The measurement probe with the update's access pattern runs on device
    segments (and writes its trivial results over the states), from the
    gradients at R = 4 and from the context's stored g_bar at R = 8, and
    refuses host memory; a device step after it is still exact."""
    n = 3 * TILE + 8
    masters, grads = rand_inputs([n], R, 1, seed=131)
    dev = DevState(masters, R)
    dev.set_grads(grads[0])
    sdp.sdp_probe_update_pattern(ctx, dev.segments(sdp), stream())
    torch.cuda.synchronize()
    assert not np.array_equal(dev.host().master[0], masters[0])
    after = DevState(masters, R)
    after.set_grads(grads[0])
    hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=1)
    norm = sdp.sdp_agg_adam_step(ctx, after.segments(sdp), hs, 0, stream(), want_norm=True)
    ref = oracle.State(masters)
    _, onorm = oracle.step(ref, grads[0], ho)
    assert norm == onorm
    check_state(after.host(), ref)
    host = HostState(sdp, masters, R)
    try:
        with pytest.raises(sdp.SdpError) as e:
            sdp.sdp_probe_update_pattern(ctx, host.segments(), stream())
        assert e.value.status == sdp.SDP_ERR_NOT_DEVICE_MEMORY
    finally:
        host.close()


def test_norm_pattern_probe(sdp, ctx):
    """The measurement probe with the g_bar-storing norm pass's access pattern
    runs on a device segment's gradients, leaves the states and the gradients
    alone, and a device step after it on the same context is still exact."""
    n, R = 3 * TILE + 8, 8
    masters, grads = rand_inputs([n], R, 1, seed=137)
    dev = DevState(masters, R)
    dev.set_grads(grads[0])
    before = dev.host()
    sdp.sdp_probe_norm_pattern(ctx, dev.segments(sdp), stream())
    torch.cuda.synchronize()
    assert states_equal(dev.host(), before)
    hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=1)
    norm = sdp.sdp_agg_adam_step(ctx, dev.segments(sdp), hs, 0, stream(), want_norm=True)
    ref = oracle.State(masters)
    _, onorm = oracle.step(ref, grads[0], ho)
    assert norm == onorm
    check_state(dev.host(), ref)
    host = HostState(sdp, masters, R)
    try:
        with pytest.raises(sdp.SdpError) as e:
            sdp.sdp_probe_norm_pattern(ctx, host.segments(), stream())
        assert e.value.status == sdp.SDP_ERR_NOT_DEVICE_MEMORY
    finally:
        host.close()


@pytest.mark.parametrize("chunk_tiles", [1, 2, 4])
def test_streamed_matches_oracle_and_device(sdp, ctx, ctx_poison, ctx_nostore, chunk_tiles):
    sizes = [3 * TILE + 5, 1, 70000]
    R = 3
    steps = 2
    masters, grads = rand_inputs(sizes, R, steps, seed=21 + chunk_tiles)
    log(f"streamed chunk={chunk_tiles} tiles")
    hps = [hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t) for t in range(1, steps + 1)]
    dev = DevState(masters, R)
    ref = oracle.State(masters)
    dev_states, ref_states, norms = [], [], []
    for t in range(steps):
        dnorm = dev_step(sdp, ctx, dev, grads[t], hps[t][0])
        _, onorm = oracle.step(ref, grads[t], hps[t][1])
        check_norm(dnorm, onorm)
        dev_states.append(dev.host())
        ref_states.append(ref.copy())
        norms.append(dnorm)
    for c in (ctx_poison, ctx_nostore):
        host = HostState(sdp, masters, R)
        try:
            for t in range(steps):
                host.set_grads(grads[t])
                snorm = sdp.sdp_stream_step(c, host.segments(), hps[t][0], chunk_tiles * TILE)
                assert snorm == norms[t], "streamed norm differs from device norm"
                got = host.host()
                check_state(got, ref_states[t])
                assert states_equal(got, dev_states[t]), "streamed differs from device mode"
        finally:
            host.close()


@pytest.mark.parametrize("R", [1, 5, 8, 16])
@pytest.mark.parametrize("flags", ["plain", "gbar_never", "staged"])
def test_streamed_ranks_equal_device_mode(sdp, ctx, R, flags):
    """Streamed mode over the rank counts the slot layout depends on (the
    norm pass's R arrays back to back, the update's R gradient arrays when
    g_bar is not kept), with the slots poisoned: device mode's bits."""
    sizes = [2 * TILE + 7, 33]
    masters, grads = rand_inputs(sizes, R, 2, seed=171 + R)
    f = sdp.SDP_FLAG_DEBUG_POISON | {"plain": 0, "gbar_never": sdp.SDP_FLAG_STREAM_GBAR_NEVER,
                                     "staged": sdp.SDP_FLAG_STREAM_STAGED}[flags]
    c = sdp.sdp_ctx_create(0, TILE, 16, f)
    dev = DevState(masters, R)
    host = PageableState(sdp, masters, R) if flags == "staged" else HostState(sdp, masters, R)
    try:
        for t in (1, 2):
            hs = sdp.make_params(lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t)
            dn = dev_step(sdp, ctx, dev, grads[t - 1], hs)
            host.set_grads(grads[t - 1])
            sn = sdp.sdp_stream_step(c, host.segments(), hs, TILE)
            assert sn == dn
            assert states_equal(host.host(), dev.host()), f"R={R} {flags} step {t}"
    finally:
        host.close()
        sdp.sdp_ctx_destroy(c)


@pytest.mark.parametrize("staged", [False, True])
def test_d2h_copy_kernel_equals_runtime_copies(sdp, ctx, staged, monkeypatch):
    """Device-to-host copies through the library's copy kernel (every copy,
    or those of at most the default 64 MiB) and through the runtime give the
    same bits, with ragged byte counts (odd element counts of BF16) and one
    to three chunks per segment, pinned and staged, with the slot poisoning
    on; all equal device mode."""
    sizes = [3 * TILE + 5, 1, 70001, 2 * TILE]
    R = 2
    masters, grads = rand_inputs(sizes, R, 2, seed=151 + int(staged))
    dev = DevState(masters, R)
    hps = [sdp.make_params(lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t) for t in (1, 2)]
    dev_states, dev_norms = [], []
    for t in (1, 2):
        dev_norms.append(dev_step(sdp, ctx, dev, grads[t - 1], hps[t - 1]))
        dev_states.append(dev.host())
    flags = sdp.SDP_FLAG_DEBUG_POISON | (sdp.SDP_FLAG_STREAM_STAGED if staged else 0)
    for limit in ("0", None, str(1 << 40)):
        if limit is None:
            monkeypatch.delenv("SDP_D2H_KERNEL_MAX_BYTES", raising=False)
        else:
            monkeypatch.setenv("SDP_D2H_KERNEL_MAX_BYTES", limit)
        c = sdp.sdp_ctx_create(0, 2 * TILE, R, flags)  # reads the variable
        host = (PageableState if staged else HostState)(sdp, masters, R)
        try:
            for t in (1, 2):
                host.set_grads(grads[t - 1])
                n = sdp.sdp_stream_step(c, host.segments(), hps[t - 1], 2 * TILE)
                assert n == dev_norms[t - 1]
                assert states_equal(host.host(), dev_states[t - 1]), f"limit {limit} step {t}"
        finally:
            host.close()
            sdp.sdp_ctx_destroy(c)
    monkeypatch.delenv("SDP_D2H_KERNEL_MAX_BYTES", raising=False)


@pytest.mark.parametrize("staged", [False, True])
@pytest.mark.parametrize("chunk_tiles", [1, 2])
def test_streamed_host_cast_equals_device_mode(sdp, ctx, staged, chunk_tiles):
    """SDP_FLAG_STREAM_HOST_CAST: the BF16 parameters are rounded on the host
    from the returned master instead of crossing the link.  Pinned and
    staged, with slot poisoning, ragged sizes and several chunks per segment,
    every output equals device mode bit for bit, and param_bf16 =
    bf16(master)."""
    sizes = [3 * TILE + 5, 1, 70001, 2 * TILE]
    R = 3
    masters, grads = rand_inputs(sizes, R, 2, seed=171 + chunk_tiles + 10 * int(staged))
    dev = DevState(masters, R)
    hps = [sdp.make_params(lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t) for t in (1, 2)]
    want = []
    for t in (1, 2):
        n = dev_step(sdp, ctx, dev, grads[t - 1], hps[t - 1])
        want.append((n, dev.host()))
    flags = sdp.SDP_FLAG_STREAM_HOST_CAST | sdp.SDP_FLAG_DEBUG_POISON | (sdp.SDP_FLAG_STREAM_STAGED if staged else 0)
    c = sdp.sdp_ctx_create(0, chunk_tiles * TILE, R, flags)
    host = (PageableState if staged else HostState)(sdp, masters, R)
    try:
        for t in (1, 2):
            host.set_grads(grads[t - 1])
            n = sdp.sdp_stream_step(c, host.segments(), hps[t - 1], chunk_tiles * TILE)
            assert n == want[t - 1][0]
            got = host.host()
            assert states_equal(got, want[t - 1][1]), f"step {t}"
            for s in range(len(sizes)):
                assert np.array_equal(got.param_bf16[s], oracle.bf16(got.master[s]))
    finally:
        host.close()
        sdp.sdp_ctx_destroy(c)


def test_staged_copy_threads_do_not_change_results(sdp, ctx, monkeypatch):
    """The staged mode's cap on copy threads while transfers are in flight
    (one thread, two, the default four, sixteen) is a schedule only: every
    cap gives device mode's bits, over five chunks per step."""
    sizes = [5 * TILE + 9]
    R = 3
    masters, grads = rand_inputs(sizes, R, 2, seed=163)
    dev = DevState(masters, R)
    hps = [sdp.make_params(lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t) for t in (1, 2)]
    want = []
    for t in (1, 2):
        n = dev_step(sdp, ctx, dev, grads[t - 1], hps[t - 1])
        want.append((n, dev.host()))
    for threads in ("1", "2", None, "16"):
        if threads is None:
            monkeypatch.delenv("SDP_STAGED_COPY_THREADS", raising=False)
        else:
            monkeypatch.setenv("SDP_STAGED_COPY_THREADS", threads)
        c = sdp.sdp_ctx_create(0, TILE, R, sdp.SDP_FLAG_STREAM_STAGED | sdp.SDP_FLAG_DEBUG_POISON)
        host = PageableState(sdp, masters, R)
        try:
            for t in (1, 2):
                host.set_grads(grads[t - 1])
                n = sdp.sdp_stream_step(c, host.segments(), hps[t - 1], TILE)
                assert n == want[t - 1][0]
                assert states_equal(host.host(), want[t - 1][1]), f"{threads} copy threads, step {t}"
        finally:
            host.close()
            sdp.sdp_ctx_destroy(c)
    monkeypatch.delenv("SDP_STAGED_COPY_THREADS", raising=False)


@pytest.fixture(scope="module")
def ctx_staged(sdp):
    c = sdp.sdp_ctx_create(0, 4 * TILE, 16, sdp.SDP_FLAG_STREAM_STAGED | sdp.SDP_FLAG_DEBUG_POISON)
    yield c
    sdp.sdp_ctx_destroy(c)


@pytest.fixture(scope="module")
def ctx_staged_nostore(sdp):
    c = sdp.sdp_ctx_create(0, 2 * TILE, 8, sdp.SDP_FLAG_STREAM_STAGED | sdp.SDP_FLAG_STREAM_GBAR_NEVER)
    yield c
    sdp.sdp_ctx_destroy(c)


@pytest.mark.parametrize("chunk_tiles", [1, 2])
def test_staged_streamed_matches_device_and_oracle(sdp, ctx, ctx_staged, ctx_staged_nostore, chunk_tiles):
    """Staged streamed mode on pageable (and on pinned) host memory gives the
    same bits as device mode, and matches the oracle."""
    sizes = [3 * TILE + 5, 1, 70000, 2 * TILE]
    R = 3
    steps = 3
    masters, grads = rand_inputs(sizes, R, steps, seed=61 + chunk_tiles)
    hps = [hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t) for t in range(1, steps + 1)]
    dev = DevState(masters, R)
    ref = oracle.State(masters)
    dev_states, ref_states, norms = [], [], []
    for t in range(steps):
        norms.append(dev_step(sdp, ctx, dev, grads[t], hps[t][0]))
        oracle.step(ref, grads[t], hps[t][1])
        dev_states.append(dev.host())
        ref_states.append(ref.copy())
    for c in (ctx_staged, ctx_staged_nostore):
        for host in (PageableState(sdp, masters, R), HostState(sdp, masters, R)):
            for t in range(steps):
                host.set_grads(grads[t])
                snorm = sdp.sdp_stream_step(c, host.segments(), hps[t][0], chunk_tiles * TILE)
                assert snorm == norms[t]
                got = host.host()
                check_state(got, ref_states[t])
                assert states_equal(got, dev_states[t]), f"staged streamed differs from device mode at step {t + 1}"
            host.close()
    # the staged mode still refuses device memory
    with pytest.raises(sdp.SdpError) as e:
        sdp.sdp_stream_step(ctx_staged, dev.segments(sdp), hps[0][0], TILE)
    assert e.value.status == sdp.SDP_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("sizes", [[5], [TILE + 3], [TILE, 7], [2 * TILE + 1, TILE]])
def test_staged_streamed_few_chunks(sdp, ctx, ctx_staged, sizes):
    """One to four chunks: the staged mode's moves out of its outgoing bounce
    buffers finish every chunk, the last one included, and equal device
    mode."""
    R = 2
    masters, grads = rand_inputs(sizes, R, 2, seed=71 + len(sizes))
    dev = DevState(masters, R)
    host = PageableState(sdp, masters, R)
    try:
        for t in (1, 2):
            hs = sdp.make_params(lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t)
            dn = dev_step(sdp, ctx, dev, grads[t - 1], hs)
            host.set_grads(grads[t - 1])
            sn = sdp.sdp_stream_step(ctx_staged, host.segments(), hs, TILE)
            assert sn == dn
            assert states_equal(host.host(), dev.host()), f"step {t}"
    finally:
        host.close()


@pytest.mark.parametrize("mode", ["host_cast", "device_cast"])
def test_deliver_params(sdp, ctx, mode):
    """Parameter delivery: the device BF16 window equals bf16(host master),
    for pinned and pageable masters, ragged sizes and both chunkings."""
    m = sdp.SDP_DELIVER_HOST_CAST if mode == "host_cast" else sdp.SDP_DELIVER_DEVICE_CAST
    rng = np.random.default_rng(77)
    for n in (1, 7, TILE + 3, 3 * TILE + 5, 1 << 20):
        x = (rng.normal(0, 0.02, n) * np.exp2(rng.integers(-20, 20, n))).astype(np.float32)
        x[:min(n, 3)] = [np.nan, np.inf, -0.0][:min(n, 3)]
        want = oracle.bf16(x)
        hb = sdp.HostBuffer(max(16, 4 * n))
        pinned = hb.view(np.float32, n)
        pinned[:] = x
        for src in (x, pinned):
            for chunk in (TILE, 2 * TILE):
                out = torch.full((n,), 0x5555, dtype=torch.int16, device="cuda")
                sdp.sdp_deliver_params(ctx, src.ctypes.data, out.data_ptr(), n, chunk, m)
                assert np.array_equal(out.cpu().numpy().view(np.uint16), want), (n, chunk, src is pinned)


def test_grad_norm_modes_agree(sdp, ctx):
    sizes = [TILE * 2 + 1, 513]
    R = 5
    _, grads = rand_inputs(sizes, R, 1, seed=33)
    dev = DevState([np.zeros(n, np.float32) for n in sizes], R)
    dev.set_grads(grads[0])
    dn = sdp.sdp_grad_norm(ctx, dev.segments(sdp), True, 0, stream())
    host = HostState(sdp, [np.zeros(n, np.float32) for n in sizes], R)
    try:
        host.set_grads(grads[0])
        hn = sdp.sdp_grad_norm(ctx, host.segments(), False, TILE)
    finally:
        host.close()
    on = oracle.grad_norm(grads[0])
    check_norm(dn, on)
    assert dn == hn
    # the staged context takes pageable gradients
    staged = sdp.sdp_ctx_create(0, TILE, R, sdp.SDP_FLAG_STREAM_STAGED)
    pg = PageableState(sdp, [np.zeros(n, np.float32) for n in sizes], R)
    try:
        pg.set_grads(grads[0])
        assert sdp.sdp_grad_norm(staged, pg.segments(), False, TILE) == dn
    finally:
        pg.close()
        sdp.sdp_ctx_destroy(staged)


def test_norm_equals_exactly_rounded_sum(sdp, ctx):
    """The GPU's double-double norm equals the oracle's exactly rounded one,
    bit for bit, in both modes, on gradients of widely spread magnitude."""
    rng = np.random.default_rng(123)
    for trial in range(12):
        R = int(rng.integers(1, 9))
        sizes = [int(rng.integers(1, 3 * TILE)) for _ in range(int(rng.integers(1, 4)))]
        grads = []
        for n in sizes:
            gs = []
            for r in range(R):
                x = rng.normal(0, 1, n) * np.exp2(rng.integers(-60, 60, n).astype(np.float64))
                gs.append(synth.to_bf16_bits(x.astype(np.float32)))
            grads.append(gs)
        want = oracle.grad_norm(grads)
        dev = DevState([np.zeros(n, np.float32) for n in sizes], R)
        dev.set_grads(grads)
        got = sdp.sdp_grad_norm(ctx, dev.segments(sdp), True, 0, stream())
        host = HostState(sdp, [np.zeros(n, np.float32) for n in sizes], R)
        host.set_grads(grads)
        got_s = sdp.sdp_grad_norm(ctx, host.segments(), False, TILE)
        assert got == want and got_s == want, (trial, got, got_s, want)


@pytest.mark.parametrize("mode", ["device", "streamed", "staged", "host_cast"])
@pytest.mark.parametrize("bad", [np.nan, np.inf])
def test_nonfinite_gradient_leaves_states_unchanged(sdp, ctx, mode, bad):
    sizes = [TILE + 9]
    R = 2
    masters, grads = rand_inputs(sizes, R, 1, seed=44)
    g = [[x.copy() for x in grads[0][0]]]
    g[0][1][12345] = synth.to_bf16_bits(np.array([bad], np.float32))[0]
    hs = sdp.make_params(step=1)
    if mode == "device":
        dev = DevState(masters, R)
        dev.pb[0].fill_(7)
        before = dev.host()
        with pytest.raises(sdp.SdpNonFinite) as e:
            dev_step(sdp, ctx, dev, g, hs)
        assert not np.isfinite(e.value.norm)
        assert states_equal(before, dev.host())
        # without a norm request the call is asynchronous and still skips the update
        dev_step(sdp, ctx, dev, g, hs, want_norm=False)
        assert states_equal(before, dev.host())
        norm, clip, nonfinite = sdp.sdp_ctx_last_norm(ctx)
        assert nonfinite and not np.isfinite(norm)
    else:
        flags = {"streamed": 0, "staged": sdp.SDP_FLAG_STREAM_STAGED, "host_cast": sdp.SDP_FLAG_STREAM_HOST_CAST}[mode]
        c = sdp.sdp_ctx_create(0, TILE, R, flags) if flags else ctx
        host = (PageableState if mode == "staged" else HostState)(sdp, masters, R)
        try:
            host.pb[0][:] = 7
            host.set_grads(g)
            before = host.host()
            with pytest.raises(sdp.SdpNonFinite):
                sdp.sdp_stream_step(c, host.segments(), hs, TILE)
            assert states_equal(before, host.host())
            # the context still works afterwards
            host.set_grads(grads[0])
            sdp.sdp_stream_step(c, host.segments(), hs, TILE)
            assert not states_equal(before, host.host())
        finally:
            host.close()
            if c is not ctx:
                sdp.sdp_ctx_destroy(c)


def test_argument_errors_have_no_side_effects(sdp, ctx):
    n, R = 4096, 2
    masters, grads = rand_inputs([n], R, 1, seed=55)
    dev = DevState(masters, R)
    dev.set_grads(grads[0])
    torch.cuda.synchronize()
    before = dev.host()
    hs = sdp.make_params(step=1)
    S = sdp.segments_from_tensors

    def expect(status, segs, params=hs, chunk=0):
        with pytest.raises(sdp.SdpError) as e:
            sdp.sdp_agg_adam_step(ctx, segs, params, chunk, stream(), want_norm=True)
        assert e.value.status == status, (e.value.name, e.value.detail)

    p, m, v, pb, g = dev.p[0], dev.m[0], dev.v[0], dev.pb[0], dev.g[0]
    expect(sdp.SDP_ERR_ALIGNMENT, S([(p[1:], m[1:], v[1:], pb[1:], [x[1:] for x in g])]))
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, [])]))                 # R = 0
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, g * 9)]))              # R = 18
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, [p.view(torch.int16)[:n], g[1]])]))  # grad aliases master
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, p, v, pb, g)]))                  # master aliases exp_avg
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, g)]), params=sdp.make_params(step=0))
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, g)]), params=sdp.make_params(beta1=1.0, step=1))
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, g)]), chunk=1000)
    expect(sdp.SDP_ERR_INVALID_ARGUMENT, S([(p, m, v, pb, g), (p, m, v, pb, g[:1])]))  # R differs
    host = np.zeros(n, np.float32)
    expect(sdp.SDP_ERR_NOT_DEVICE_MEMORY,
           sdp.Segments([(host.ctypes.data, m.data_ptr(), v.data_ptr(), pb.data_ptr(), [x.data_ptr() for x in g], n)]))
    expect(sdp.SDP_ERR_NOT_DEVICE_MEMORY,
           sdp.Segments([(p.data_ptr(), m.data_ptr(), v.data_ptr(), pb.data_ptr(), [x.data_ptr() for x in g],
                          1 << 34)]))                                            # far beyond the allocation
    # streamed mode: device or pageable pointers are not pinned; chunk bounds
    with pytest.raises(sdp.SdpError) as e:
        sdp.sdp_stream_step(ctx, S([(p, m, v, pb, g)]), hs, TILE)
    assert e.value.status == sdp.SDP_ERR_NOT_PINNED
    hm = [np.zeros(n, np.float32) for _ in range(3)]
    hb = [np.zeros(n, np.uint16) for _ in range(3)]
    pageable = sdp.Segments([(hm[0].ctypes.data, hm[1].ctypes.data, hm[2].ctypes.data, hb[0].ctypes.data,
                              [hb[1].ctypes.data, hb[2].ctypes.data], n)])
    with pytest.raises(sdp.SdpError) as e:
        sdp.sdp_stream_step(ctx, pageable, hs, TILE)
    assert e.value.status == sdp.SDP_ERR_NOT_PINNED
    with pytest.raises(sdp.SdpError) as e:
        sdp.sdp_stream_step(ctx, pageable, hs, 8 * TILE)
    assert e.value.status == sdp.SDP_ERR_CHUNK_TOO_LARGE
    # the host-rounding and staged flags need streamed-mode staging
    for flag in (sdp.SDP_FLAG_STREAM_HOST_CAST, sdp.SDP_FLAG_STREAM_STAGED):
        with pytest.raises(sdp.SdpError) as e:
            sdp.sdp_ctx_create(0, 0, 2, flag)
        assert e.value.status == sdp.SDP_ERR_INVALID_ARGUMENT
    torch.cuda.synchronize()
    assert states_equal(before, dev.host())


def test_cast_bf16_exhaustive(sdp, ctx):
    """The device BF16 re-emit over all 2^32 FP32 bit patterns, against the oracle."""
    chunk = 1 << 28
    src = torch.empty(chunk, dtype=torch.int32, device="cuda")
    dst = torch.empty(chunk, dtype=torch.int16, device="cuda")
    base = torch.arange(chunk, dtype=torch.int64, device="cuda")
    bad = 0
    for k in range((1 << 32) // chunk):
        vals = base + k * chunk
        vals = torch.where(vals >= (1 << 31), vals - (1 << 32), vals)
        src.copy_(vals.to(torch.int32))
        sdp.sdp_cast_bf16(ctx, src.data_ptr(), dst.data_ptr(), chunk, stream())
        got = dst.cpu().numpy().view(np.uint16)
        f = src.cpu().numpy().view(np.float32)
        bad += int(np.count_nonzero(got != oracle.bf16(f)))
        if k % 4 == 0:
            log(f"cast chunk {k}")
    assert bad == 0
    # ragged sizes
    for n in (1, 7, 9, 1000003):
        x = torch.randn(n, device="cuda")
        y = torch.empty(n, dtype=torch.int16, device="cuda")
        sdp.sdp_cast_bf16(ctx, x.data_ptr(), y.data_ptr(), n, stream())
        assert np.array_equal(y.cpu().numpy().view(np.uint16), oracle.bf16(x.cpu().numpy()))


# ---------------------------------------------------------------------------
# The mean gradient's single rounding, on rank sets built to make it hard

def mean_edge_grads(R, n, seed):
    """Ordinary N(0, 1e-3) BF16 gradients with mean_cases' stress sets written
    over scattered elements, the last one (the ragged tail) included."""
    import mean_cases
    _, grads = rand_inputs([n], R, 1, seed=seed)
    g = np.stack(grads[0][0])
    sets = [mean_cases.wide_span(R, 400, seed=R)]
    if R >= 3:
        sets.append(mean_cases.near_midpoint(R, 600, seed=50 + R))
    sets.append(mean_cases.subnormal_remainder(R))
    special = np.concatenate(sets, axis=1)
    rng = np.random.default_rng(seed)
    pos = np.append(rng.choice(n - 1, special.shape[1] - 1, replace=False), n - 1)
    g[:, pos] = special
    return [[g[r].copy() for r in range(R)]]


@pytest.mark.parametrize("R", [2, 3, 5, 8, 11, 13, 16])
def test_mean_exact_quotient_edge_cases(sdp, ctx, ctx_store, ctx_nostore, R):
    """With beta1 = 0 and no clipping, exp_avg after one step is the mean
    gradient itself, so every mode's g_bar is compared with the oracle's bit
    for bit (the oracle's mean is pinned to fractions.Fraction), and the whole
    step with the oracle's by the usual criteria."""
    n = 3 * TILE + 5
    log(f"mean edge cases R={R}")
    masters, _ = rand_inputs([n], R, 1, seed=300 + R)
    grads = mean_edge_grads(R, n, seed=400 + R)
    want = oracle.mean_grads(grads[0])
    hs, ho = hp_pair(sdp, lr=1e-3, beta1=0.0, weight_decay=0.01, max_grad_norm=0.0, step=1)
    ref = oracle.State(masters)
    rc, onorm = oracle.step(ref, grads, ho)
    assert rc == oracle.ORC_OK

    def check(state, norm, what):
        check_norm(norm, onorm)
        assert norm == onorm, f"{what}: norm {norm!r} != exactly rounded {onorm!r}"
        bad = np.flatnonzero(state.exp_avg[0].view(np.uint32) != want.view(np.uint32))
        assert bad.size == 0, (f"{what}: g_bar differs on {bad.size} elements, first at {bad[0]}: "
                               f"gpu {state.exp_avg[0][bad[0]]!r} oracle {want[bad[0]]!r} "
                               f"ranks {[hex(int(x[bad[0]])) for x in grads[0]]}")
        check_state(state, ref)

    for c, what in ((ctx, "device"), (ctx_store, "device, stored g_bar"), (ctx_nostore, "device, no g_bar")):
        dev = DevState(masters, R)
        norm = dev_step(sdp, c, dev, grads, hs)
        check(dev.host(), norm, what)
    # streamed, pinned, in chunks of one tile
    hst = HostState(sdp, masters, R)
    try:
        hst.set_grads(grads)
        norm = sdp.sdp_stream_step(ctx, hst.segments(), hs, TILE)
        check(hst.host(), norm, "streamed")
    finally:
        hst.close()
    # host-update route, FP32 mean gradient
    from test_gpu_host_route import RouteState
    st = RouteState(sdp, masters, R)
    try:
        st.set_grads(grads)
        norm = sdp.sdp_host_update_step(ctx, st.segments(sdp), hs, 2 * TILE, sdp.SDP_GBAR_F32)
        check(st.state(), norm, "host route")
    finally:
        st.close()
