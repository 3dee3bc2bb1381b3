// C ABI of libsdp, streamed mode (sdp_stream_step): states live in pinned
// host memory (or, staged, in any host memory) and move through two device
// staging slots.  A copy stream carries host-to-device copies; a compute
// stream runs the kernels and the device-to-host copies.  Events h2d_done[s]
// and slot_free[s] order each slot's reuse: a slot is refilled only after
// its previous consumer finished (the paper's buffer-reuse rule, Design,
// completion and buffer reuse), and the update of a chunk starts as soon as
// its copy has landed (chunked overlap within a layer).  Phase 1 streams the
// gradients for the global norm; phase 2 streams master/m/v through the
// fused update and back.
#include "sdp_rt.h"
#include "sdp_schedule.h"

namespace sdprt {

// Device -> pinned host copies (dst[k] <- src[k], bytes[k]) on stream st:
// those of at most d2h_kernel_max bytes (16-byte aligned) as one
// launch of the library's copy kernel, the others as runtime copies.  The
// kernel stores through the device's mapping of the host memory, as the
// runtime reports it: the same address for hipHostMalloc memory, possibly
// another for registered memory; memory without one takes a runtime copy.
// (The same kernel measured slower than the runtime's host-to-device copies
// at every chunk size, so those stay runtime copies.)  own_map: the
// destinations lie in a buffer of the context's own whose device mapping is
// offset by *own_map from its host address (looked up once, when the buffer
// was allocated), so no attribute query is needed per copy.
int d2h_copies(sdp_ctx *ctx, const std::vector<std::pair<char *, const char *>> &ends,
               const std::vector<size_t> &bytes, hipStream_t st, const ptrdiff_t *own_map) {
    sdp::CopyBatch b{};
    for (size_t k = 0; k < ends.size(); ++k) {
        char *mapped = nullptr;
        if ((int64_t)bytes[k] <= ctx->d2h_kernel_max && b.n < sdp::kCopyBatchMax) {
            hipPointerAttribute_t at;
            if (own_map)
                mapped = ends[k].first + *own_map;
            else if (hipPointerGetAttributes(&at, ends[k].first) == hipSuccess && at.type == hipMemoryTypeHost)
                mapped = (char *)at.devicePointer;
            else
                (void)hipGetLastError();
        }
        if (mapped && (((uintptr_t)mapped | (uintptr_t)ends[k].second) % 16) == 0) {
            b.dst[b.n] = mapped;
            b.src[b.n] = ends[k].second;
            b.bytes[b.n] = (int64_t)bytes[k];
            ++b.n;
        } else {
            HIP_TRY(hipMemcpyAsync(ends[k].first, ends[k].second, bytes[k], hipMemcpyDeviceToHost, st));
        }
    }
    if (b.n > 0) {
        const int per_copy = ctx->d2h_kernel_blocks > 0 ? ctx->d2h_kernel_blocks
                                                          : std::max(kD2HMinBlocksPerCopy, kD2HLaunchBlocks / b.n);
        HIP_TRY(sdp::launch_copy_batch(b, per_copy, st));
    }
    return SDP_OK;
}

namespace {

int poison(sdp_ctx *ctx, int k) {
    if (!(ctx->flags & SDP_FLAG_DEBUG_POISON)) return SDP_OK;
    HIP_TRY(sdp::launch_fill_u32(ctx->staging + (size_t)k * ctx->slot_bytes, (int64_t)(ctx->slot_bytes / 4),
                                 0xFFC0FFC0u, ctx->s_comp));
    return SDP_OK;
}

// Runs of transfers that are contiguous in the slot, for the bounce copies.
std::vector<Xfer> merge_runs(std::vector<Xfer> xs) {
    std::sort(xs.begin(), xs.end(), [](const Xfer &a, const Xfer &b) { return a.off < b.off; });
    std::vector<Xfer> runs;
    for (const Xfer &x : xs) {
        if (!runs.empty() && runs.back().off + runs.back().bytes == x.off)
            runs.back().bytes += x.bytes;
        else
            runs.push_back({x.off, nullptr, x.bytes});
    }
    return runs;
}

// Host -> slot `sl` copies of one chunk, enqueued on the copy stream.  In the
// staged mode the host threads (at most `width` of them, 0: all) first copy
// into pinned bounce buffer `bi`, after waiting for that buffer's previous
// copies to leave it.
int copy_in(sdp_ctx *ctx, int sl, int bi, const std::vector<Xfer> &xs, int width) {
    char *dev = ctx->staging + (size_t)sl * ctx->slot_bytes;
    jitter_host(ctx);
    SDP_TRY(jitter_stream(ctx, ctx->s_copy));
    if (!staged(ctx)) {
        for (const Xfer &x : xs)
            HIP_TRY(hipMemcpyAsync(dev + x.off, x.host, x.bytes, hipMemcpyHostToDevice, ctx->s_copy));
        return SDP_OK;
    }
    char *bin = ctx->bounce_in + (size_t)bi * ctx->slot_bytes;
    if (ctx->bin_used[bi]) HIP_TRY(hipEventSynchronize(ctx->bin_done[bi]));
    std::vector<Job> jobs;
    for (const Xfer &x : xs) jobs.push_back({bin + x.off, x.host, x.bytes});
    pool_jobs(ctx->copier, jobs, width);
    for (const Xfer &r : merge_runs(xs))
        HIP_TRY(hipMemcpyAsync(dev + r.off, bin + r.off, r.bytes, hipMemcpyHostToDevice, ctx->s_copy));
    HIP_TRY(hipEventRecord(ctx->bin_done[bi], ctx->s_copy));
    ctx->bin_used[bi] = true;
    return SDP_OK;
}

// Slot `sl` -> host copies of one chunk, enqueued on the compute stream.  In
// the staged mode they land in outgoing bounce buffer `bo` and are moved to
// their destinations by drain().
int copy_out(sdp_ctx *ctx, int sl, int bo, const std::vector<Xfer> &xs) {
    char *dev = ctx->staging + (size_t)sl * ctx->slot_bytes;
    std::vector<std::pair<char *, const char *>> ends;
    std::vector<size_t> bytes;
    SDP_TRY(jitter_stream(ctx, ctx->s_comp));
    if (!staged(ctx)) {
        for (const Xfer &x : xs) {
            ends.push_back({x.host, dev + x.off});
            bytes.push_back(x.bytes);
        }
        SDP_TRY(d2h_copies(ctx, ends, bytes, ctx->s_comp, nullptr));
        if (host_cast(ctx)) HIP_TRY(hipEventRecord(ctx->d2h_done[bo], ctx->s_comp));
        return SDP_OK;
    }
    char *bout = ctx->bounce_out + (size_t)bo * 14 * (size_t)ctx->max_chunk;
    for (const Xfer &r : merge_runs(xs)) {
        ends.push_back({bout + r.off, dev + r.off});
        bytes.push_back(r.bytes);
    }
    SDP_TRY(d2h_copies(ctx, ends, bytes, ctx->s_comp, &ctx->bounce_out_map));
    HIP_TRY(hipEventRecord(ctx->d2h_done[bo], ctx->s_comp));
    ctx->pending_out[bo] = xs;
    return SDP_OK;
}

// Wait for outgoing copies `bo` to land, then, on at most `width` host
// threads (0: all), move them from the bounce buffer to their host
// destinations (staged mode) and round the chunk's master to BF16
// (SDP_FLAG_STREAM_HOST_CAST).
int drain(sdp_ctx *ctx, int bo, int width) {
    if (ctx->pending_out[bo].empty() && ctx->pending_cast[bo].empty()) return SDP_OK;
    jitter_host(ctx);
    HIP_TRY(hipEventSynchronize(ctx->d2h_done[bo]));
    char *bout = ctx->bounce_out + (size_t)bo * 14 * (size_t)ctx->max_chunk;
    std::vector<Job> jobs;
    for (const Xfer &x : ctx->pending_out[bo]) jobs.push_back({x.host, bout + x.off, x.bytes});
    jobs.insert(jobs.end(), ctx->pending_cast[bo].begin(), ctx->pending_cast[bo].end());
    pool_jobs(ctx->copier, jobs, width);
    ctx->pending_out[bo].clear();
    ctx->pending_cast[bo].clear();
    return SDP_OK;
}

}  // namespace

// Phase 1: gradients in, norm partials (and stored g_bar) out, then finalize.
// The chunks are sdp_sched::norm_phase_chunk elements long, larger than the
// update's from pinned memory.  The R gradient arrays lie back to back from
// the slot's start, each on a 256-byte boundary, so a staged full chunk
// crosses the link as one run.
int stream_norm_phase(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int32_t R, const Plan &plan,
                      const std::vector<Chunk> &chunks, bool store_gbar, double max_grad_norm, bool used[2]) {
    (void)n_segs;
    for (size_t k = 0; k < chunks.size(); ++k) {
        const Chunk &c = chunks[k];
        const int sl = (int)(k & 1);
        char *base = ctx->staging + (size_t)sl * ctx->slot_bytes;
        const size_t stride = (size_t)((c.len + 127) / 128 * 128) * 2;
        if ((size_t)R * stride > ctx->slot_bytes)
            return fail(SDP_ERR_CHUNK_TOO_LARGE, "norm pass chunk of %lld elements does not fit the slot", (long long)c.len);
        std::vector<Xfer> xs;
        const uint16_t *gp[SDP_MAX_RANKS];
        for (int32_t r = 0; r < R; ++r) {
            xs.push_back({(size_t)r * stride, (char *)(segs[c.seg].grads[r] + c.off), (size_t)c.len * 2});
            gp[r] = (const uint16_t *)(base + (size_t)r * stride);
        }
        if (used[sl]) HIP_TRY(hipStreamWaitEvent(ctx->s_copy, ctx->slot_free[sl], 0));
        SDP_TRY(copy_in(ctx, sl, (int)(k % kInBufs), xs, 0));
        HIP_TRY(hipEventRecord(ctx->h2d_done[sl], ctx->s_copy));
        HIP_TRY(hipStreamWaitEvent(ctx->s_comp, ctx->h2d_done[sl], 0));
        SDP_TRY(jitter_stream(ctx, ctx->s_comp));
        SDP_TRY(norm_launch(ctx, R, gp, c.len, tile_partials(ctx, plan.tile_base[c.seg] + c.off / SDP_NORM_TILE),
                            store_gbar ? ctx->gbar + plan.gbar_base[c.seg] + c.off : nullptr, ctx->s_comp));
        SDP_TRY(poison(ctx, sl));
        HIP_TRY(hipEventRecord(ctx->slot_free[sl], ctx->s_comp));
        used[sl] = true;
    }
    return finalize_launch(ctx, plan.tiles, max_grad_norm, ctx->s_comp);
}

namespace {

// Phase 2: master/m/v in (and the gradients again unless g_bar is stored),
// fused update, master/m/v and BF16 parameters back out (or, with
// SDP_FLAG_STREAM_HOST_CAST, the BF16 parameters rounded on the host from the
// returned master).  Chunk j uses slot (j + k0) mod 2, continuing phase 1's
// alternation.  Staged or rounding on the host, the host thread stages and
// enqueues chunk j + kStageAhead before it drains chunk j.  While
// copies are in flight the host copies run on staged_copy_threads threads:
// more of them starve the device-to-host copies of host memory (phase 1,
// with the link busy in one direction only, is not hurt and uses them all).
// The first chunk's staging and the last chunk's drain have the link to
// themselves and use every thread.
int stream_update_phase(sdp_ctx *ctx, const sdp_segment *segs, int32_t R, const Plan &plan,
                        const std::vector<Chunk> &chunks, bool stored_gbar, const sdp_adamw_params *hp, bool used[2],
                        size_t k0) {
    auto issue = [&](size_t j) -> int {
        const Chunk &c = chunks[j];
        const sdp_segment &g = segs[c.seg];
        const int sl = (int)((j + k0) & 1);
        Slot slot = slot_at(ctx, sl);
        const size_t f4 = (size_t)c.len * 4, b2 = (size_t)c.len * 2;
        std::vector<Xfer> in = {{off_in_slot(ctx, sl, slot.p), (char *)(g.master + c.off), f4},
                                {off_in_slot(ctx, sl, slot.m), (char *)(g.exp_avg + c.off), f4},
                                {off_in_slot(ctx, sl, slot.v), (char *)(g.exp_avg_sq + c.off), f4}};
        if (!stored_gbar)
            for (int32_t r = 0; r < R; ++r)
                in.push_back({off_in_slot(ctx, sl, slot.g[r]), (char *)(g.grads[r] + c.off), b2});
        if (used[sl]) HIP_TRY(hipStreamWaitEvent(ctx->s_copy, ctx->slot_free[sl], 0));
        SDP_TRY(copy_in(ctx, sl, (int)((j + k0) % kInBufs), in, j == 0 ? 0 : ctx->staged_copy_threads));
        HIP_TRY(hipEventRecord(ctx->h2d_done[sl], ctx->s_copy));
        HIP_TRY(hipStreamWaitEvent(ctx->s_comp, ctx->h2d_done[sl], 0));
        const uint16_t *gp[SDP_MAX_RANKS];
        for (int32_t r = 0; r < R; ++r) gp[r] = slot.g[r];
        SDP_TRY(jitter_stream(ctx, ctx->s_comp));
        SDP_TRY(update_launch(ctx, R, hp, slot.p, slot.m, slot.v, slot.pb, gp,
                              stored_gbar ? ctx->gbar + plan.gbar_base[c.seg] + c.off : nullptr, c.len, ctx->s_comp));
        std::vector<Xfer> out = {{off_in_slot(ctx, sl, slot.p), (char *)(g.master + c.off), f4},
                                 {off_in_slot(ctx, sl, slot.m), (char *)(g.exp_avg + c.off), f4},
                                 {off_in_slot(ctx, sl, slot.v), (char *)(g.exp_avg_sq + c.off), f4}};
        const int bo = (int)(j % kOutBufs);
        if (host_cast(ctx)) {
            // the master's rounding, from where it lands on the host
            const void *src = staged(ctx) ? (const void *)(ctx->bounce_out + (size_t)bo * 14 * (size_t)ctx->max_chunk +
                                                           off_in_slot(ctx, sl, slot.p))
                                          : (const void *)(g.master + c.off);
            ctx->pending_cast[bo] = {{g.param_bf16 + c.off, src, (size_t)c.len, Job::kCastBf16}};
        } else {
            out.push_back({off_in_slot(ctx, sl, slot.pb), (char *)(g.param_bf16 + c.off), b2});
        }
        SDP_TRY(copy_out(ctx, sl, bo, out));
        SDP_TRY(poison(ctx, sl));
        HIP_TRY(hipEventRecord(ctx->slot_free[sl], ctx->s_comp));
        used[sl] = true;
        return SDP_OK;
    };
    if (!staged(ctx) && !host_cast(ctx)) {
        for (size_t j = 0; j < chunks.size(); ++j) SDP_TRY(issue(j));
        return SDP_OK;
    }
    size_t next = 0;
    for (size_t j = 0; j < chunks.size(); ++j) {
        for (; next < chunks.size() && next <= j + kStageAhead; ++next) SDP_TRY(issue(next));
        SDP_TRY(drain(ctx, (int)(j % kOutBufs), j + 1 == chunks.size() ? 0 : ctx->staged_copy_threads));
    }
    return SDP_OK;
}

}  // namespace

}  // namespace sdprt

using namespace sdprt;

extern "C" {

int sdp_stream_step(sdp_ctx *ctx, const sdp_segment *host_segs, int32_t n_segs, const sdp_adamw_params *hp,
                    int64_t chunk_elems, double *grad_norm_out) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    SDP_TRY(check_hparams(hp));
    DeviceGuard guard(ctx->device);
    int32_t R = 0;
    SDP_TRY(stream_common_checks(ctx, host_segs, n_segs, chunk_elems, false, &R));
    const Plan plan = make_plan(host_segs, n_segs);
    const bool store = !(ctx->flags & SDP_FLAG_STREAM_GBAR_NEVER);
    SDP_TRY(ensure_partials(ctx, plan.tiles));
    if (store) SDP_TRY(ensure_gbar(ctx, plan.gbar_elems));
    const std::vector<Chunk> chunks = make_chunks(host_segs, n_segs, chunk_elems);
    const std::vector<Chunk> norm_chunks =
        make_chunks(host_segs, n_segs, sdp_sched::norm_phase_chunk(chunk_elems, R, staged(ctx)));
    SDP_TRY(order_after_last(ctx, ctx->s_copy));
    SDP_TRY(order_after_last(ctx, ctx->s_comp));
    bool used[2] = {false, false};
    int rc = stream_norm_phase(ctx, host_segs, n_segs, R, plan, norm_chunks, store, hp->max_grad_norm, used);
    NormState st{};
    if (rc == SDP_OK) rc = read_norm(ctx, ctx->s_comp, &st);
    if (rc != SDP_OK) {
        (void)sync_streams(ctx);
        return rc;
    }
    if (grad_norm_out) *grad_norm_out = st.norm;
    if (st.nonfinite) {
        SDP_TRY(sync_streams(ctx));
        SDP_TRY(mark_done(ctx, ctx->s_comp));
        return fail(SDP_ERR_NONFINITE, "gradient norm is not finite (%g); nothing was updated", st.norm);
    }
    rc = stream_update_phase(ctx, host_segs, R, plan, chunks, store, hp, used, norm_chunks.size());
    int rc2 = sync_streams(ctx);
    // after a failure, results still waiting in bounce buffers belong to this
    // call only: never let a later call move them
    for (auto &xs : ctx->pending_out) xs.clear();
    for (auto &js : ctx->pending_cast) js.clear();
    if (rc != SDP_OK) return rc;
    if (rc2 != SDP_OK) return rc2;
    return mark_done(ctx, ctx->s_comp);
}

}  // extern "C"
