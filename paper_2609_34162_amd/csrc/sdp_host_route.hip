// C ABI of libsdp, the host lanes: parameter delivery (sdp_deliver_params,
// sdp_cast_bf16_host) and the host-update route (sdp_host_update_step,
// sdp_host_adamw).  In the route the gradients stay in device memory; the
// GPU computes the norm and, piece by piece, the mean gradient, which the
// copy stream moves into pinned stage buffers while the host threads run
// AdamW on the states in host memory.
#include "sdp_rt.h"
#include "sdp_schedule.h"

namespace sdprt {
namespace {

sdp_host::AdamConsts host_consts(const sdp_adamw_params *hp, double clip) {
    sdp::UpdateArgs u{};
    fill_consts(hp, u);
    sdp_host::AdamConsts k;
    k.c = clip;
    k.lr_wd = u.lr_wd;
    k.beta1 = u.beta1;
    k.one_minus_beta1 = u.one_minus_beta1;
    k.beta2 = u.beta2;
    k.one_minus_beta2 = u.one_minus_beta2;
    k.step_size = u.step_size;
    k.inv_bc2 = u.inv_bc2;
    k.eps = u.eps;
    return k;
}

// Instruction set of the host update: the CPU's best unless SDP_HOST_SIMD=0.
int host_simd() {
    if (const char *env = std::getenv("SDP_HOST_SIMD"))
        if (std::atoi(env) == 0) return sdp_host::kScalar;
    return sdp_host::simd_best();
}

// Host AdamW over n elements, in 32,768-element pieces over the pool's
// threads (on the calling thread alone when pool is NULL).
void host_adamw(HostPool *pool, const sdp_host::AdamArgs &a, const sdp_host::AdamConsts &k, int64_t n) {
    constexpr int64_t kPiece = 32768;
    const int simd = host_simd();
    const size_t pieces = (size_t)cdiv(n, kPiece);
    auto body = [&](size_t j) {
        const int64_t i0 = (int64_t)j * kPiece;
        sdp_host::adamw_range(a, k, i0, std::min(n, i0 + kPiece), simd);
    };
    if (pool)
        pool->run(pieces, body);
    else
        for (size_t j = 0; j < pieces; ++j) body(j);
}

// The host-update route over validated segments (grads in device memory,
// states in host memory).  Phase 1: the norm pass over the device gradients
// and the finalize; the norm state comes back to the host.  Phase 2, piece
// by piece: the GPU writes g_bar of piece j (FP32 or BF16) into device slot
// j%2 on the compute stream, the copy stream moves it into pinned host buffer
// j%2, and the host threads update piece j-1 from the other buffer meanwhile.
// The pieces grow from C/16 to C over the call's start (route_pieces).
int host_route(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int32_t R, const Plan &plan,
               const sdp_adamw_params *hp, int64_t C, bool bf16, double *grad_norm_out) {
    hipStream_t sc = ctx->s_comp, sy = ctx->s_copy;
    SDP_TRY(device_norm(ctx, segs, n_segs, R, plan, false, hp->max_grad_norm, sc));
    NormState st{};
    SDP_TRY(read_norm(ctx, sc, &st));
    if (grad_norm_out) *grad_norm_out = st.norm;
    if (st.nonfinite) return fail(SDP_ERR_NONFINITE, "gradient norm is not finite (%g); nothing was updated", st.norm);
    const sdp_host::AdamConsts k = host_consts(hp, st.clip);
    // pieces of at most C elements, growing from C/16 so that the host
    // threads start after a short first copy and each copy hides behind the
    // host update of the piece before it
    std::vector<Chunk> chunks;
    {
        std::vector<int64_t> numels;
        for (int32_t k = 0; k < n_segs; ++k) numels.push_back(segs[k].numel);
        for (const sdp_sched::RoutePiece &pc : sdp_sched::route_pieces(numels, C))
            chunks.push_back({pc.seg, pc.off, pc.len});
    }
    const size_t esz = bf16 ? 2 : 4;
    bool used[2] = {false, false};
    auto issue = [&](size_t j) -> int {
        const Chunk &c = chunks[j];
        const int sl = (int)(j & 1);
        char *dev = ctx->staging + (size_t)sl * ctx->slot_bytes;
        char *host = ctx->stage + (size_t)sl * stage_bytes(ctx);
        // the slot's previous copy to the host has read it
        if (used[sl]) HIP_TRY(hipStreamWaitEvent(sc, ctx->slot_free[sl], 0));
        sdp::GbarArgs a{};
        for (int32_t r = 0; r < R; ++r) a.g[r] = segs[c.seg].grads[r] + c.off;
        a.n = c.len;
        a.out = dev;
        a.bf16 = bf16 ? 1 : 0;
        SDP_TRY(jitter_stream(ctx, sc));
        hipEvent_t t0 = timed_begin(ctx, sc);
        HIP_TRY(sdp::launch_gbar_out(R, a, sc));
        timed_end(ctx, sc, t0, kGbar, c.len);
        // h2d_done doubles as "g_bar of this slot is written" here
        HIP_TRY(hipEventRecord(ctx->h2d_done[sl], sc));
        HIP_TRY(hipStreamWaitEvent(sy, ctx->h2d_done[sl], 0));
        SDP_TRY(jitter_stream(ctx, sy));
        SDP_TRY(d2h_copies(ctx, {{host, dev}}, {(size_t)c.len * esz}, sy, &ctx->stage_map));
        HIP_TRY(hipEventRecord(ctx->slot_free[sl], sy));  // in the host buffer; the slot is free
        used[sl] = true;
        return SDP_OK;
    };
    if (!chunks.empty()) SDP_TRY(issue(0));
    for (size_t j = 0; j < chunks.size(); ++j) {
        // the next chunk's kernel and copy run while the host updates this one
        const Clock::time_point ti = Clock::now();
        if (j + 1 < chunks.size()) SDP_TRY(issue(j + 1));
        const int sl = (int)(j & 1);
        jitter_host(ctx);
        const Clock::time_point t0 = Clock::now();
        HIP_TRY(hipEventSynchronize(ctx->slot_free[sl]));
        const Clock::time_point t1 = Clock::now();
        const Chunk &c = chunks[j];
        const sdp_segment &g = segs[c.seg];
        sdp_host::AdamArgs a;
        a.p = g.master + c.off;
        a.m = g.exp_avg + c.off;
        a.v = g.exp_avg_sq + c.off;
        a.pb = g.param_bf16 + c.off;
        a.gbar = ctx->stage + (size_t)sl * stage_bytes(ctx);
        a.gbar_bf16 = bf16 ? 1 : 0;
        host_adamw(ctx->copier, a, k, c.len);
        if (ctx->timing) {
            const Clock::time_point t2 = Clock::now();
            ctx->host_wait_ms += ms_between(t0, t1);
            if (j + 1 < chunks.size()) {
                ctx->host_issue_ms += ms_between(ti, t0);
                ctx->host_issues += 1;
            }
            ctx->host_adam_ms += ms_between(t1, t2);
            ctx->host_adam_elems += c.len;
        }
    }
    return SDP_OK;
}

}  // namespace
}  // namespace sdprt

using namespace sdprt;

extern "C" {

int sdp_cast_bf16_host(sdp_ctx *ctx, const float *src, uint16_t *dst, int64_t n) {
    t_err.clear();
    if (!src || !dst || n < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_cast_bf16_host: bad argument");
    if (ctx && ctx->copier)
        pool_jobs(ctx->copier, {{dst, src, (size_t)n, Job::kCastBf16}});
    else
        cast_bf16_host(src, dst, (size_t)n);
    return SDP_OK;
}

}  // extern "C"

namespace {

// Parameter delivery; with `gate` the call returns once every chunk is
// enqueued and `consumer` waits for the last copy on the GPU, else it
// blocks until the copies have landed.
int deliver(sdp_ctx *ctx, const float *host_master, uint16_t *dev_bf16, int64_t n, int64_t chunk_elems, int mode,
            bool gate, hipStream_t consumer) {
    if (!ctx || !host_master || !dev_bf16 || n < 1)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_deliver_params: bad argument");
    if (mode != SDP_DELIVER_HOST_CAST && mode != SDP_DELIVER_DEVICE_CAST)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_deliver_params: unknown mode %d", mode);
    if (!ctx->staging) return fail(SDP_ERR_CHUNK_TOO_LARGE, "context was created without streamed-mode staging");
    SDP_TRY(check_chunk(chunk_elems, false));
    if (chunk_elems > ctx->max_chunk)
        return fail(SDP_ERR_CHUNK_TOO_LARGE, "chunk_elems %lld exceeds the context's %lld", (long long)chunk_elems,
                    (long long)ctx->max_chunk);
    if (!aligned(host_master) || !aligned(dev_bf16))
        return fail(SDP_ERR_ALIGNMENT, "sdp_deliver_params: pointers must be %d-byte aligned", SDP_ALIGN);
    DeviceGuard guard(ctx->device);
    SDP_TRY(check_host_ptr(host_master, "host_master", 0));
    SDP_TRY(check_device_ptr(ctx, dev_bf16, (size_t)n * 2, "dev_bf16", 0));
    const bool pinned = is_pinned_host(host_master);
    if (mode == SDP_DELIVER_HOST_CAST || !pinned) SDP_TRY(ensure_host_stage(ctx));
    SDP_TRY(order_after_last(ctx, ctx->s_copy));
    SDP_TRY(order_after_last(ctx, ctx->s_comp));
    bool used[2] = {false, false};
    int rc = SDP_OK;
    size_t k = 0;
    for (int64_t off = 0; off < n && rc == SDP_OK; off += chunk_elems, ++k) {
        const int sl = (int)(k & 1);
        const int64_t len = std::min(chunk_elems, n - off);
        char *bin = ctx->stage ? ctx->stage + (size_t)sl * stage_bytes(ctx) : nullptr;
        jitter_host(ctx);
        if ((rc = jitter_stream(ctx, ctx->s_copy)) != SDP_OK) break;
        if (mode == SDP_DELIVER_HOST_CAST) {
            // host threads round chunk k while the DMA still moves chunk k-1
            if (ctx->stage_used[sl] && hipEventSynchronize(ctx->h2d_done[sl]) != hipSuccess) {
                rc = fail(SDP_ERR_HIP, "sdp_deliver_params: event wait failed");
                break;
            }
            pool_jobs(ctx->copier, {{bin, host_master + off, (size_t)len, Job::kCastBf16}});
            if (hipMemcpyAsync(dev_bf16 + off, bin, (size_t)len * 2, hipMemcpyHostToDevice, ctx->s_copy) != hipSuccess ||
                hipEventRecord(ctx->h2d_done[sl], ctx->s_copy) != hipSuccess)
                rc = fail(SDP_ERR_HIP, "sdp_deliver_params: copy enqueue failed");
            ctx->stage_used[sl] = true;
        } else {
            Slot slot = slot_at(ctx, sl);
            std::vector<Xfer> xs = {{off_in_slot(ctx, sl, slot.p), (char *)(host_master + off), (size_t)len * 4}};
            if (used[sl] && hipStreamWaitEvent(ctx->s_copy, ctx->slot_free[sl], 0) != hipSuccess) {
                rc = fail(SDP_ERR_HIP, "sdp_deliver_params: stream wait failed");
                break;
            }
            if (pinned) {
                if (hipMemcpyAsync(slot.p, host_master + off, (size_t)len * 4, hipMemcpyHostToDevice, ctx->s_copy) !=
                    hipSuccess)
                    rc = fail(SDP_ERR_HIP, "sdp_deliver_params: copy enqueue failed");
            } else {
                if (ctx->stage_used[sl] && hipEventSynchronize(ctx->h2d_done[sl]) != hipSuccess) {
                    rc = fail(SDP_ERR_HIP, "sdp_deliver_params: event wait failed");
                    break;
                }
                pool_jobs(ctx->copier, {{bin, host_master + off, (size_t)len * 4}});
                if (hipMemcpyAsync(slot.p, bin, (size_t)len * 4, hipMemcpyHostToDevice, ctx->s_copy) != hipSuccess)
                    rc = fail(SDP_ERR_HIP, "sdp_deliver_params: copy enqueue failed");
                ctx->stage_used[sl] = true;
            }
            if (rc != SDP_OK) break;
            if (hipEventRecord(ctx->h2d_done[sl], ctx->s_copy) != hipSuccess ||
                hipStreamWaitEvent(ctx->s_comp, ctx->h2d_done[sl], 0) != hipSuccess ||
                jitter_stream(ctx, ctx->s_comp) != SDP_OK ||
                sdp::launch_cast_bf16(slot.p, dev_bf16 + off, len, ctx->s_comp) != hipSuccess ||
                hipEventRecord(ctx->slot_free[sl], ctx->s_comp) != hipSuccess)
                rc = fail(SDP_ERR_HIP, "sdp_deliver_params: enqueue failed");
            used[sl] = true;
        }
    }
    if (!gate || rc != SDP_OK) {
        const std::string err = t_err;
        const int rc2 = sync_streams(ctx);
        if (rc != SDP_OK) {
            t_err = err;
            return rc;
        }
        if (rc2 != SDP_OK) return rc2;
        return mark_done(ctx, ctx->s_comp);
    }
    // the version gate: last_done follows this call's work on both streams,
    // and the consumer's later work follows last_done
    HIP_TRY(hipEventRecord(ctx->copy_done, ctx->s_copy));
    HIP_TRY(hipStreamWaitEvent(ctx->s_comp, ctx->copy_done, 0));
    SDP_TRY(mark_done(ctx, ctx->s_comp));
    HIP_TRY(hipStreamWaitEvent(consumer, ctx->last_done, 0));
    return SDP_OK;
}

}  // namespace

extern "C" {

int sdp_deliver_params(sdp_ctx *ctx, const float *host_master, uint16_t *dev_bf16, int64_t n, int64_t chunk_elems,
                       int mode) {
    t_err.clear();
    return deliver(ctx, host_master, dev_bf16, n, chunk_elems, mode, false, nullptr);
}

int sdp_deliver_params_async(sdp_ctx *ctx, const float *host_master, uint16_t *dev_bf16, int64_t n,
                             int64_t chunk_elems, int mode, void *consumer_stream) {
    t_err.clear();
    return deliver(ctx, host_master, dev_bf16, n, chunk_elems, mode, true, (hipStream_t)consumer_stream);
}

int sdp_host_update_step(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, const sdp_adamw_params *hp,
                         int64_t chunk_elems, int gbar_format, double *grad_norm_out) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    SDP_TRY(check_hparams(hp));
    if (gbar_format != SDP_GBAR_F32 && gbar_format != SDP_GBAR_BF16)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_host_update_step: unknown gradient format %d", gbar_format);
    if (!ctx->staging) return fail(SDP_ERR_CHUNK_TOO_LARGE, "context was created without streamed-mode staging");
    SDP_TRY(check_chunk(chunk_elems, false));
    if (chunk_elems > ctx->max_chunk)
        return fail(SDP_ERR_CHUNK_TOO_LARGE, "chunk_elems %lld exceeds the context's %lld", (long long)chunk_elems,
                    (long long)ctx->max_chunk);
    DeviceGuard guard(ctx->device);
    int32_t R = 0;
    SDP_TRY(validate_segments(ctx, segs, n_segs, kAnyHost, kDeviceMem, false, &R));
    const Plan plan = make_plan(segs, n_segs);
    SDP_TRY(ensure_partials(ctx, plan.tiles));
    SDP_TRY(ensure_host_stage(ctx));
    SDP_TRY(order_after_last(ctx, ctx->s_comp));
    SDP_TRY(order_after_last(ctx, ctx->s_copy));
    const int rc = host_route(ctx, segs, n_segs, R, plan, hp, chunk_elems, gbar_format == SDP_GBAR_BF16,
                              grad_norm_out);
    // nothing of this call may still read the caller's gradients on return
    const std::string err = t_err;
    const int rc2 = sync_streams(ctx);
    if (rc != SDP_OK) {
        t_err = err;
        return rc;
    }
    if (rc2 != SDP_OK) return rc2;
    return mark_done(ctx, ctx->s_comp);
}

int sdp_host_adamw(sdp_ctx *ctx, float *master, float *exp_avg, float *exp_avg_sq, uint16_t *param_bf16,
                   const void *gbar, int gbar_format, int64_t n, double clip_coef, const sdp_adamw_params *hp) {
    t_err.clear();
    if (!master || !exp_avg || !exp_avg_sq || !param_bf16 || !gbar || n < 1)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_host_adamw: NULL buffer or n < 1");
    if (gbar_format != SDP_GBAR_F32 && gbar_format != SDP_GBAR_BF16)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_host_adamw: unknown gradient format %d", gbar_format);
    if (!std::isfinite(clip_coef) || clip_coef < 0.0)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_host_adamw: clip_coef must be finite and >= 0");
    SDP_TRY(check_hparams(hp));
    const size_t gb = (size_t)n * (gbar_format == SDP_GBAR_BF16 ? 2 : 4);
    const Range rs[5] = {{(uintptr_t)master, (uintptr_t)master + (size_t)n * 4, 0, "master"},
                         {(uintptr_t)exp_avg, (uintptr_t)exp_avg + (size_t)n * 4, 0, "exp_avg"},
                         {(uintptr_t)exp_avg_sq, (uintptr_t)exp_avg_sq + (size_t)n * 4, 0, "exp_avg_sq"},
                         {(uintptr_t)param_bf16, (uintptr_t)param_bf16 + (size_t)n * 2, 0, "param_bf16"},
                         {(uintptr_t)gbar, (uintptr_t)gbar + gb, 0, "gbar"}};
    for (int x = 0; x < 5; ++x) {
        if (rs[x].a % SDP_ALIGN != 0)
            return fail(SDP_ERR_ALIGNMENT, "sdp_host_adamw: %s is not %d-byte aligned", rs[x].what, SDP_ALIGN);
        for (int y = 0; y < x; ++y)
            if (overlap(rs[x], rs[y]))
                return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_host_adamw: %s overlaps %s", rs[x].what, rs[y].what);
    }
    if (ctx && !ctx->copier) ctx->copier = new_pool(ctx, default_host_threads());
    sdp_host::AdamArgs a;
    a.p = master;
    a.m = exp_avg;
    a.v = exp_avg_sq;
    a.pb = param_bf16;
    a.gbar = gbar;
    a.gbar_bf16 = gbar_format == SDP_GBAR_BF16 ? 1 : 0;
    host_adamw(ctx ? ctx->copier : nullptr, a, host_consts(hp, clip_coef), n);
    return SDP_OK;
}

int sdp_ctx_set_host_threads(sdp_ctx *ctx, int32_t threads) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    if (threads < 1 || threads > 256)
        return fail(SDP_ERR_INVALID_ARGUMENT, "host threads must be in 1..256 (got %d)", threads);
    delete ctx->copier;
    ctx->copier = new_pool(ctx, threads);
    return SDP_OK;
}

int sdp_ctx_host_threads(sdp_ctx *ctx, int32_t *threads_out) {
    t_err.clear();
    if (!ctx || !threads_out) return fail(SDP_ERR_INVALID_ARGUMENT, "context or out is NULL");
    *threads_out = ctx->copier ? ctx->copier->size() : default_host_threads();
    return SDP_OK;
}

}  // extern "C"
