"""The step-time model (sdp_predict_step, sdp_tune_chunk) against closed
forms of its dependency recurrence and its resource bound.  Host code only:
runs without a GPU."""
import math

import numpy as np
import pytest

TILE = 65536


@pytest.fixture(scope="module")
def sdp():
    from paper_2609_34162_amd import sdp as mod
    return mod


def rates(sdp, **kw):
    # host memory so fast that the DMA never slows a host task, unless a test says otherwise
    base = dict(h2d_gbs=50.0, d2h_gbs=40.0, both_gbs=90.0, copy_cmd_us=0.0, norm_gbs=5000.0, update_gbs=4000.0,
                launch_us=0.0, sync_us=0.0, host_gbs=1e7, host_task_us=0.0, host_adam_gbs=300.0)
    base.update(kw)
    return sdp.make_rates(**base)


def us(nbytes, gbs):
    return nbytes / (gbs * 1e3)


def test_streamed_single_chunk_is_the_serial_sum(sdp):
    """One chunk: nothing can overlap, so the recurrence is the sum of every
    node's duration, command costs included."""
    N, R = 3 * TILE + 5, 3
    r = dict(copy_cmd_us=7.0, launch_us=3.0, sync_us=11.0)
    rt = rates(sdp, **r)
    got = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, 4 * TILE, 0, rt)
    want = (R * 7.0 + us(2 * R * N, 50.0)            # gradients in
            + us((2 * R + 4) * N, 5000.0) + 3.0      # norm pass, storing g_bar
            + 3.0 + 11.0                             # finalize, read-back
            + 3 * 7.0 + us(12 * N, 50.0)             # states in
            + us(30 * N, 4000.0) + 3.0               # update from stored g_bar
            + 1 * 7.0 + us(14 * N, 40.0))            # results out: every copy at most 64 MiB, one kernel launch
    assert math.isclose(got.predicted_ms, want / 1e3, rel_tol=1e-12)
    assert got.n_chunks == 1
    # without stored g_bar the gradients cross twice and the update reads them
    got2 = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, 4 * TILE, sdp.SDP_FLAG_STREAM_GBAR_NEVER, rt)
    want2 = (want - us(4 * N, 5000.0) + R * 7.0 + us(2 * R * N, 50.0) - us(30 * N, 4000.0)
             + us((26 + 2 * R) * N, 4000.0))
    assert math.isclose(got2.predicted_ms, want2 / 1e3, rel_tol=1e-12)


@pytest.mark.parametrize("issue_us", [0.0, 29.0])
def test_host_route_two_segments_closed_form(sdp, issue_us):
    sizes, R = [TILE + 1, 2 * TILE], 4
    rt = rates(sdp, copy_cmd_us=5.0, launch_us=2.0, sync_us=13.0, host_task_us=17.0, host_issue_us=issue_us)
    for sched, esz in ((sdp.SDP_SCHED_HOST_ROUTE_F32, 4), (sdp.SDP_SCHED_HOST_ROUTE_BF16, 2)):
        got = sdp.sdp_predict_step(sched, sizes, R, 4 * TILE, 0, rt)
        want = sum(us(2 * R * n, 5000.0) + 2.0 for n in sizes) + 2.0 + 13.0
        # two chunks (one per segment): kernel and copy of the second overlap
        # the host update of the first
        g = [us((2 * R + esz) * n, 5000.0) + 2.0 for n in sizes]
        c = [5.0 + us(esz * n, 40.0) for n in sizes]
        h = [us((26 + esz) * n, 300.0) + 17.0 for n in sizes]
        # the host thread enqueues chunk 1 (issue_us) right after the read-back
        t_c0 = want + g[0] + c[0]
        t_h0 = max(want + issue_us, t_c0 + 13.0) + h[0]   # the host learns of a copy's end sync_us later
        t_c1 = max(want + issue_us + g[1], want + g[0] + g[1], t_c0) + c[1]
        total = max(t_h0, t_c1 + 13.0) + h[1]
        assert math.isclose(got.predicted_ms, total / 1e3, rel_tol=1e-12), sched


def test_two_chunk_phase_two_recurrence(sdp):
    """Two chunks without link contention (both_gbs = h2d + d2h): phase two is
    the recurrence with fixed durations: in_0, then upd_0 and out_0 on the
    compute stream while in_1 runs on the copy stream, then upd_1, out_1."""
    N, R = 2 * TILE, 2
    rt = rates(sdp, both_gbs=90.0, launch_us=1.0)
    got = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, TILE, 0, rt).predicted_ms * 1e3
    L = TILE
    # phase one moves only the gradients, in chunks that fill the slot laid
    # out for L elements: floor((14 + 2R) / 2R) = 4 tiles here, so one chunk
    n1 = us(2 * R * N, 50.0) + us((2 * R + 4) * N, 5000.0) + 1.0
    t1 = n1 + 1.0  # finalize; read-back costs nothing here
    a = us(12 * L, 50.0)
    u = us(30 * L, 4000.0) + 1.0
    d = us(14 * L, 40.0)
    # in_1 and out_0 overlap but both_gbs = h2d + d2h, so neither slows down
    t2 = max(2 * a, a + u + d) + u + d
    assert math.isclose(got, t1 + t2, rel_tol=1e-12)
    # an event between the copy and the compute stream takes effect dep_us
    # later: each kernel after its copy; host edges (the read-back) do not pay it
    e = 23.0
    got_e = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, TILE, 0,
                                 rates(sdp, both_gbs=90.0, launch_us=1.0, dep_us=e)).predicted_ms * 1e3
    t1e = n1 + e + 1.0
    t2e = max(2 * a + e, a + e + u + d) + u + d
    assert math.isclose(got_e, t1e + t2e, rel_tol=1e-12)


def test_norm_pass_chunks_fill_the_slot(sdp):
    """From pinned memory, phase one moves only the R gradient arrays, in
    chunks that fill the slot the update pass lays out for the call's chunk
    C: the largest tile multiple of (14 + 2R) C / 2R elements.  With the link and the kernels
    free, a step costs its copy commands: R per phase-one chunk, then three
    per update chunk on the copy stream, and the last chunk's copy-kernel
    launch."""
    fast = dict(h2d_gbs=1e12, d2h_gbs=1e12, both_gbs=2e12, norm_gbs=1e12, update_gbs=1e12, copy_cmd_us=5.0)
    # (R, C, N, phase-one chunks): 2.75 C -> 2 tiles; 8 C; 3.75 C -> 3 tiles
    for R, C, N, n1 in ((4, TILE, 8 * TILE, 4), (1, TILE, 16 * TILE, 2), (8, 2 * TILE, 8 * TILE, 3)):
        n2 = N // C
        got = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, C, 0, rates(sdp, **fast))
        assert got.n_chunks == n2
        assert math.isclose(got.predicted_ms * 1e3, (n1 * R + 3 * n2 + 1) * 5.0, rel_tol=1e-4), (R, C)
    # staged, phase one keeps the update's chunk, and a full chunk crosses as
    # one run each way: 8 + 8 copies in and the last chunk's launch out
    st = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED_STAGED, [8 * TILE], 4, TILE, 0, rates(sdp, **fast))
    assert math.isclose(st.predicted_ms * 1e3, 17 * 5.0, rel_tol=1e-4)


def test_link_contention_slows_overlapping_copies(sdp):
    N, R = 8 * TILE, 2
    free = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, TILE, 0, rates(sdp, both_gbs=90.0))
    shared = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, TILE, 0, rates(sdp, both_gbs=60.0))
    assert shared.predicted_ms > free.predicted_ms
    # never slower than running every copy and kernel one after another
    serial = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, 8 * TILE, 0, rates(sdp, both_gbs=60.0))
    assert shared.predicted_ms <= serial.predicted_ms * (1 + 1e-12) + 1e-9
    assert shared.link_ms > free.link_ms


def test_bound_never_exceeds_prediction(sdp):
    rng = np.random.default_rng(3)
    for trial in range(200):
        sizes = [int(x) for x in rng.integers(1, 40 * TILE, int(rng.integers(1, 4)))]
        R = int(rng.integers(1, 17))
        chunk = TILE * int(rng.integers(1, 9))
        h2d, d2h = rng.uniform(5, 80, 2)
        rt = rates(sdp, h2d_gbs=h2d, d2h_gbs=d2h, both_gbs=rng.uniform(max(h2d, d2h), h2d + d2h),
                   copy_cmd_us=rng.uniform(0, 30), norm_gbs=rng.uniform(100, 8000),
                   update_gbs=rng.uniform(100, 8000), launch_us=rng.uniform(0, 10), sync_us=rng.uniform(0, 50),
                   host_gbs=rng.uniform(10, 500), host_task_us=rng.uniform(0, 50),
                   host_adam_gbs=rng.uniform(10, 500))
        sched = int(rng.integers(0, 4))
        flags = sdp.SDP_FLAG_STREAM_GBAR_NEVER if rng.random() < 0.3 else 0
        p = sdp.sdp_predict_step(sched, sizes, R, chunk, flags, rt)
        assert p.bound_ms == max(p.h2d_ms, p.d2h_ms, p.link_ms, p.gpu_ms, p.host_ms, p.dram_ms)
        assert p.bound_ms <= p.predicted_ms * (1 + 1e-9), (trial, sched, p.bound_ms, p.predicted_ms)
        assert p.n_chunks == sum(-(-n // chunk) for n in sizes)


@pytest.mark.parametrize("kappa", [1.0, 2.5])
def test_host_update_shares_host_memory_with_the_copy(sdp, kappa):
    """Host route, two equal chunks: the update of chunk 0 starts with the
    copy of chunk 1 and runs at min(its own rate, host_gbs - kappa * copy
    rate) until that copy ends, then at its own rate; kappa is the host
    memory a host task loses per DMA byte."""
    L, R = 4 * TILE, 2
    A, B = 300.0, 320.0   # the AdamW lane's own rate; host memory bandwidth
    rt = rates(sdp, host_gbs=B, host_adam_gbs=A, norm_gbs=1e9, dma_host_cost=kappa)
    esz = 2
    got = sdp.sdp_predict_step(sdp.SDP_SCHED_HOST_ROUTE_BF16, [2 * L], R, L, 0, rt).predicted_ms * 1e3
    start = us(2 * R * 2 * L, 1e9) + us((2 * R + esz) * L, 1e9)   # norm pass, first mean-gradient kernel
    c = us(esz * L, 40.0)                     # one copy, alone on the link
    W = (26 + esz) * L                        # host bytes of one chunk's update
    # the second kernel ran long ago (its rate is huge), so copy 1 starts with update 0
    slow = min(A, B - kappa * 40.0) * 1e3     # bytes per us while copy 1 runs
    done_during = slow * c
    assert done_during < W
    u0 = c + (W - done_during) / (A * 1e3)
    want = start + c + u0 + W / (A * 1e3)     # update 1 follows update 0 with the link idle
    assert math.isclose(got, want, rel_tol=1e-9), (got, want)
    p = sdp.sdp_predict_step(sdp.SDP_SCHED_HOST_ROUTE_BF16, [2 * L], R, L, 0, rt)
    assert math.isclose(p.dram_ms, (2 * W + 2 * esz * L) / (B * 1e9) * 1e3, rel_tol=1e-12)


def test_streamed_host_cast_single_chunk_closed_form(sdp):
    """One chunk with the BF16 parameters rounded on the host: 12 B per
    element come back in one copy-kernel launch, then one host task reads
    the master and writes the BF16 parameters (6 B per element), alone on
    host memory."""
    N, R = 3 * TILE + 5, 3
    rt = rates(sdp, copy_cmd_us=7.0, launch_us=3.0, sync_us=11.0, host_gbs=100.0, host_task_us=5.0)
    got = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, 4 * TILE, sdp.SDP_FLAG_STREAM_HOST_CAST, rt)
    want = (R * 7.0 + us(2 * R * N, 50.0) + us((2 * R + 4) * N, 5000.0) + 3.0 + 3.0 + 11.0
            + 3 * 7.0 + us(12 * N, 50.0) + us(30 * N, 4000.0) + 3.0
            + 1 * 7.0 + us(12 * N, 40.0)             # master, m, v out
            + 11.0 + 5.0 + us(6 * N, 100.0))         # host rounding, once the host learns the copy ended
    assert math.isclose(got.predicted_ms, want / 1e3, rel_tol=1e-12)
    plain = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, 4 * TILE, 0, rt)
    assert math.isclose(got.d2h_ms, plain.d2h_ms * 12 / 14, rel_tol=1e-12)
    assert math.isclose(got.h2d_ms, plain.h2d_ms, rel_tol=1e-12)


def test_streamed_host_cast_many_chunks(sdp):
    """Many chunks: with fast host lanes, rounding on the host beats copying
    the BF16 parameters back (fewer link bytes); with slow ones it loses."""
    sizes, R, C = [40 * TILE + 3], 4, 4 * TILE
    fast = rates(sdp, host_gbs=1e6, host_task_us=0.0)
    plain = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, sizes, R, C, 0, fast)
    hc = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, sizes, R, C, sdp.SDP_FLAG_STREAM_HOST_CAST, fast)
    assert hc.predicted_ms < plain.predicted_ms
    assert hc.bound_ms <= hc.predicted_ms
    slow = rates(sdp, host_gbs=2.0, host_task_us=0.0)
    hc_slow = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, sizes, R, C, sdp.SDP_FLAG_STREAM_HOST_CAST, slow)
    assert hc_slow.predicted_ms > plain.predicted_ms


def test_staged_equals_plain_when_host_lanes_are_free(sdp):
    # R = 16: (14 + 2R) C / 2R rounds down to C, so both modes chunk phase one alike
    N, R = 10 * TILE + 3, 16
    rt = rates(sdp, host_gbs=1e9, host_task_us=0.0)
    a = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, [N], R, 2 * TILE, 0, rt)
    b = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED_STAGED, [N], R, 2 * TILE, 0, rt)
    assert math.isclose(a.predicted_ms, b.predicted_ms, rel_tol=1e-6)
    slow = sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED_STAGED, [N], R, 2 * TILE, 0, rates(sdp, host_gbs=20.0))
    assert slow.predicted_ms > a.predicted_ms


def test_tune_chunk_is_the_argmin(sdp):
    sizes, R = [300 * TILE], 4
    cands = [TILE * k for k in (1, 2, 4, 8, 16, 32, 64)]
    for kw, expect_largest in ((dict(copy_cmd_us=2000.0), True), (dict(norm_gbs=20.0, update_gbs=20.0), False)):
        rt = rates(sdp, **kw)
        best, ms = sdp.sdp_tune_chunk(sdp.SDP_SCHED_STREAMED, sizes, R, 0, rt, cands)
        direct = [sdp.sdp_predict_step(sdp.SDP_SCHED_STREAMED, sizes, R, c, 0, rt).predicted_ms for c in cands]
        assert ms == direct
        assert best == cands[int(np.argmin(direct))]
        if expect_largest:
            assert best == cands[-1]          # per-command costs dominate: fewest chunks
        else:
            assert best < cands[-1]           # slow kernels: pipelining pays


def test_model_argument_errors(sdp):
    L = sdp._lib
    rt = rates(sdp)
    out = sdp.sdp_prediction()
    import ctypes
    arr = (ctypes.c_int64 * 1)(TILE)
    assert L.sdp_predict_step(9, arr, 1, 2, TILE, 0, rt, out) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_predict_step(0, arr, 1, 0, TILE, 0, rt, out) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_predict_step(0, arr, 1, 2, TILE + 1, 0, rt, out) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_predict_step(0, None, 1, 2, TILE, 0, rt, out) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_predict_step(0, arr, 1, 2, TILE, 0, rates(sdp, h2d_gbs=0.0), out) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_predict_step(0, arr, 1, 2, TILE, 0, rates(sdp, sync_us=float("nan")), out) == \
        sdp.SDP_ERR_INVALID_ARGUMENT
    assert L.sdp_predict_step(0, arr, 1, 2, TILE, 0, rates(sdp, dep_us=-1.0), out) == sdp.SDP_ERR_INVALID_ARGUMENT
    # host route pieces with a chunk near the int64 limit: the ramp still ends at the segment
    top = (2 ** 63 - 1) // TILE * TILE
    ok = sdp.sdp_predict_step(sdp.SDP_SCHED_HOST_ROUTE_F32, [TILE << 46], 2, top, 0, rt)
    assert math.isfinite(ok.predicted_ms) and ok.predicted_ms > 0
    # a chunk far beyond any slot: one chunk, as any chunk of at least the segment
    huge = sdp.sdp_predict_step(0, [TILE], 16, TILE << 45, 0, rt)
    assert math.isclose(huge.predicted_ms, sdp.sdp_predict_step(0, [TILE], 16, TILE, 0, rt).predicted_ms,
                        rel_tol=1e-12)
    big = (ctypes.c_int64 * 1)(TILE << 23)
    assert L.sdp_predict_step(0, big, 1, 2, TILE, 0, rt, out) == sdp.SDP_ERR_INVALID_ARGUMENT
    assert "too many" in sdp.sdp_last_error()
    best = ctypes.c_int64()
    cands = (ctypes.c_int64 * 2)(TILE, 5)
    assert L.sdp_tune_chunk(0, arr, 1, 2, 0, rt, cands, 2, ctypes.byref(best), None) == sdp.SDP_ERR_INVALID_ARGUMENT
