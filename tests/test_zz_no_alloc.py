"""sdp_agg_adam_step_noalloc: device mode with no allocation, its workspace
in the library's static device array.  Through the C ABI, against the
context's sdp_agg_adam_step (bit for bit) and the oracle, on two calls in a
row of which the second is smaller (the array keeps the first call's
contents), and on the Qwen2.5-72B layer at full size (877,674,496 params,
R = 8: 13,393 norm tiles of the array's 16,384).  The size limit is checked
before anything touches a GPU."""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import DevState, check_norm, check_state, hp_pair, log, need_gpu, rand_inputs, states_equal, torch

TILE = 65536


def test_rejects_more_tiles_than_its_workspace():
    from paper_2609_34162_amd import sdp
    per = sdp.SDP_NOALLOC_MAX_TILES * TILE // 2
    # two segments of half the limit each fit; one more element does not.
    # The limit is checked before any pointer is looked at (these are NULL).
    segs = sdp.Segments([(0, 0, 0, 0, [0, 0], per), (0, 0, 0, 0, [0, 0], per + 1)])
    with pytest.raises(sdp.SdpError) as e:
        sdp.sdp_agg_adam_step_noalloc(segs, sdp.make_params(step=1))
    assert e.value.status == sdp.SDP_ERR_INVALID_ARGUMENT and "norm tiles" in e.value.detail
    many = sdp.Segments([(0, 0, 0, 0, [0], 1)] * (sdp.SDP_NOALLOC_MAX_SEGMENTS + 1))
    with pytest.raises(sdp.SdpError) as e:
        sdp.sdp_agg_adam_step_noalloc(many, sdp.make_params(step=1))
    assert e.value.status == sdp.SDP_ERR_INVALID_ARGUMENT and "segments" in e.value.detail


@pytest.mark.gpu
def test_matches_context_step_on_two_calls_second_smaller():
    sdp = need_gpu()
    stream = torch.cuda.current_stream().cuda_stream
    ctx = sdp.sdp_ctx_create(0, 0, 16, 0)
    try:
        # the first call larger (several segments, R = 8), the second smaller
        for sizes, R, seed in (([3 * TILE + 5, 70001, 9, 2 * TILE], 8, 11), ([TILE + 3], 3, 12)):
            log(f"no-alloc step: sizes {sizes} R={R}")
            masters, grads = rand_inputs(sizes, R, 2, seed=seed)
            a, b = DevState(masters, R), DevState(masters, R)
            ref = oracle.State(masters)
            for t in (1, 2):
                hs, ho = hp_pair(sdp, lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t)
                a.set_grads(grads[t - 1])
                b.set_grads(grads[t - 1])
                n_ctx = sdp.sdp_agg_adam_step(ctx, a.segments(sdp), hs, 0, stream, want_norm=True)
                n_na = sdp.sdp_agg_adam_step_noalloc(b.segments(sdp), hs, stream, want_norm=True)
                torch.cuda.synchronize()
                _, onorm = oracle.step(ref, grads[t - 1], ho)
                assert n_na == n_ctx
                check_norm(n_na, onorm)
                assert states_equal(b.host(), a.host()), f"step {t}: differs from sdp_agg_adam_step"
                check_state(b.host(), ref)
    finally:
        sdp.sdp_ctx_destroy(ctx)


@pytest.mark.gpu
@pytest.mark.big
def test_qwen2_5_72b_layer_full_size_equals_context_step():
    sdp = need_gpu()
    stream = torch.cuda.current_stream().cuda_stream
    w = synth.workload(4)
    R = w.ranks
    log(f"no-alloc step: {w.name} N={w.numel} R={R}")
    master = synth.master(w, 0)
    grads = [[synth.grad_bf16(w, 0, 1, r) for r in range(R)]]
    a, b = DevState([master], R), DevState([master], R)
    a.set_grads(grads)
    b.set_grads(grads)
    ctx = sdp.sdp_ctx_create(0, 0, R, 0)
    try:
        hs = sdp.make_params(**w.hparams(1))
        n_ctx = sdp.sdp_agg_adam_step(ctx, a.segments(sdp), hs, w.chunk, stream, want_norm=True)
        n_na = sdp.sdp_agg_adam_step_noalloc(b.segments(sdp), hs, stream, want_norm=True)
        torch.cuda.synchronize()
        assert n_na == n_ctx
        assert states_equal(b.host(), a.host())
    finally:
        sdp.sdp_ctx_destroy(ctx)


@pytest.mark.gpu
@pytest.mark.big
def test_at_the_tile_limit_equals_context_step():
    """Exactly SDP_NOALLOC_MAX_TILES norm tiles (16,383 of one segment, whose
    last is ragged, and one of a second): the workspace's last span pairs and
    merge-stage pairs are used.  Bit for bit against sdp_agg_adam_step, two
    steps, inputs generated on the GPU."""
    sdp = need_gpu()
    stream = torch.cuda.current_stream().cuda_stream
    sizes = [(sdp.SDP_NOALLOC_MAX_TILES - 1) * TILE - 3, 3]
    R = 2
    log(f"no-alloc step at the tile limit: sizes {sizes} R={R}")
    gen = torch.Generator(device="cuda").manual_seed(5)
    grads = [[(torch.randn(n, generator=gen, device="cuda") * 1e-3).to(torch.bfloat16).view(torch.int16)
              for _ in range(R)] for n in sizes]
    masters = [torch.randn(n, generator=gen, device="cuda") * 0.02 for n in sizes]

    def fresh():
        return [(p.clone(), torch.zeros_like(p), torch.zeros_like(p), torch.zeros(p.numel(), dtype=torch.int16,
                                                                                device="cuda"), g)
                for p, g in zip(masters, grads)]

    a, b = fresh(), fresh()
    ctx = sdp.sdp_ctx_create(0, 0, R, 0)
    try:
        for t in (1, 2):
            hs = sdp.make_params(lr=1e-3, weight_decay=0.05, max_grad_norm=0.2, step=t)
            n_ctx = sdp.sdp_agg_adam_step(ctx, sdp.segments_from_tensors(a), hs, 0, stream, want_norm=True)
            n_na = sdp.sdp_agg_adam_step_noalloc(sdp.segments_from_tensors(b), hs, stream, want_norm=True)
            torch.cuda.synchronize()
            assert n_na == n_ctx, t
            for sa, sb in zip(a, b):
                for x, y in zip(sa[:4], sb[:4]):
                    assert torch.equal(x.view(torch.int32) if x.dtype == torch.float32 else x,
                                       y.view(torch.int32) if y.dtype == torch.float32 else y), f"step {t}"
    finally:
        sdp.sdp_ctx_destroy(ctx)
