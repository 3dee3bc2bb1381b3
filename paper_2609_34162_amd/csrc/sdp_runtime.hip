// C ABI of libsdp, core: errors, the context, argument validation, the
// device-mode driver, measurement support and the step-time model's entry
// points.  The streamed engine is in sdp_stream.hip, parameter delivery and
// the host-update route in sdp_host_route.hip, the kernels in
// sdp_kernels.hip, the host AdamW lane in sdp_host_adamw.cpp and the
// step-time model in sdp_schedule.cpp.
//
// Device mode (sdp_agg_adam_step): per call, one norm-partials launch per
// segment, the finalize (one launch, or two above 2,048 span partials) and
// one fused-update launch per segment, all on the caller's stream.  The clip
// coefficient stays in device memory.
#include "sdp_rt.h"
#include "sdp_schedule.h"

namespace sdprt {

thread_local std::string t_err;

int fail(int status, const char *fmt, ...) {
    char buf[1024];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    return status;
}

// Round FP32 values to BF16, nearest even, on the host (the parameter
// delivery lane, and streamed mode's host rounding): the host lanes' routine.
void cast_bf16_host(const float *src, uint16_t *dst, size_t n) { sdp_host::cast_bf16(src, dst, (int64_t)n); }

void pool_jobs(HostPool *pool, const std::vector<Job> &jobs, int width) {
    constexpr size_t kPiece = 4u << 20;      // bytes per copy piece
    constexpr size_t kCastPiece = 1u << 20;  // elements per rounding piece
    std::vector<Job> pieces;
    for (const Job &j : jobs) {
        if (j.kind == Job::kCastBf16) {
            for (size_t off = 0; off < j.bytes; off += kCastPiece)
                pieces.push_back({(uint16_t *)j.dst + off, (const float *)j.src + off,
                                  std::min(kCastPiece, j.bytes - off), Job::kCastBf16});
        } else {
            for (size_t off = 0; off < j.bytes; off += kPiece)
                pieces.push_back({(char *)j.dst + off, (const char *)j.src + off, std::min(kPiece, j.bytes - off)});
        }
    }
    pool->run(pieces.size(), [&](size_t k) {
        const Job &pc = pieces[k];
        if (pc.kind == Job::kCastBf16)
            cast_bf16_host((const float *)pc.src, (uint16_t *)pc.dst, pc.bytes);
        else
            std::memcpy(pc.dst, pc.src, pc.bytes);
    }, width);
}

// ---- validation ---------------------------------------------------------

int check_hparams(const sdp_adamw_params *hp) {
    if (!hp) return fail(SDP_ERR_INVALID_ARGUMENT, "hyperparameters are NULL");
    if (hp->step < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "step must be >= 1 (got %lld)", (long long)hp->step);
    const double v[] = {hp->lr, hp->beta1, hp->beta2, hp->eps, hp->weight_decay, hp->max_grad_norm};
    for (double x : v)
        if (!std::isfinite(x)) return fail(SDP_ERR_INVALID_ARGUMENT, "hyperparameters must be finite");
    if (hp->beta1 < 0.0 || hp->beta1 >= 1.0 || hp->beta2 < 0.0 || hp->beta2 >= 1.0)
        return fail(SDP_ERR_INVALID_ARGUMENT, "betas must lie in [0, 1)");
    if (hp->eps < 0.0) return fail(SDP_ERR_INVALID_ARGUMENT, "eps must be >= 0");
    return SDP_OK;
}

int check_device_ptr(const sdp_ctx *ctx, const void *p, size_t bytes, const char *what, int seg) {
    hipPointerAttribute_t at;
    hipError_t e = hipPointerGetAttributes(&at, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s (%p) is not device memory", seg, what, p);
    }
    if (at.type != hipMemoryTypeDevice || at.device != ctx->device)
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s (%p) is not device memory of GPU %d", seg, what, p,
                    ctx->device);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) == hipSuccess) {
        if ((const char *)p + bytes > (const char *)base + size)
            return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s: %zu bytes at %p overrun its allocation", seg, what,
                        bytes, p);
    } else {
        (void)hipGetLastError();
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s (%p): allocation range unknown", seg, what, p);
    }
    return SDP_OK;
}

int check_pinned_ptr(const void *p, size_t bytes, const char *what, int seg) {
    const void *ends[2] = {p, (const char *)p + bytes - 1};
    for (const void *q : ends) {
        hipPointerAttribute_t at;
        hipError_t e = hipPointerGetAttributes(&at, q);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(SDP_ERR_NOT_PINNED, "segment %d %s (%p, %zu bytes) is not pinned host memory", seg, what, p,
                        bytes);
        }
        if (at.type != hipMemoryTypeHost)
            return fail(SDP_ERR_NOT_PINNED, "segment %d %s (%p) is not pinned host memory", seg, what, p);
    }
    return SDP_OK;
}

// Host memory for the staged streamed mode: anything that is not device
// memory (pageable or pinned).  Pageable ranges cannot be checked further.
int check_host_ptr(const void *p, const char *what, int seg) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, p) == hipSuccess) {
        if (at.type == hipMemoryTypeDevice)
            return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d %s (%p) is device memory, not host memory", seg, what, p);
    } else {
        (void)hipGetLastError();
    }
    return SDP_OK;
}

// Checks every segment of a call; returns R and the per-segment sizes.
int validate_segments(const sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, MemKind state_kind,
                      MemKind grad_kind, bool grads_only, int32_t *R_out) {
    if (!segs || n_segs < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "need at least one segment");
    int32_t R = segs[0].n_ranks;
    if (R < 1 || R > SDP_MAX_RANKS)
        return fail(SDP_ERR_INVALID_ARGUMENT, "n_ranks must be in 1..%d (got %d)", SDP_MAX_RANKS, R);
    std::vector<Range> states, grads;
    for (int32_t s = 0; s < n_segs; ++s) {
        const sdp_segment &g = segs[s];
        if (g.n_ranks != R) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d has n_ranks %d, segment 0 has %d", s,
                                        g.n_ranks, R);
        if (g.numel < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d: numel must be >= 1", s);
        if (!g.grads) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d: grads is NULL", s);
        const int64_t n = g.numel;
        struct Buf {
            const void *p;
            size_t bytes;
            const char *what;
        };
        std::vector<Buf> bufs;
        if (!grads_only) {
            bufs.push_back({g.master, (size_t)n * 4, "master"});
            bufs.push_back({g.exp_avg, (size_t)n * 4, "exp_avg"});
            bufs.push_back({g.exp_avg_sq, (size_t)n * 4, "exp_avg_sq"});
            bufs.push_back({g.param_bf16, (size_t)n * 2, "param_bf16"});
        }
        const size_t n_state = bufs.size();
        for (int32_t r = 0; r < R; ++r) bufs.push_back({g.grads[r], (size_t)n * 2, "grad"});
        for (size_t k = 0; k < bufs.size(); ++k) {
            const Buf &b = bufs[k];
            if (!b.p) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d: %s is NULL", s, b.what);
            if (!aligned(b.p))
                return fail(SDP_ERR_ALIGNMENT, "segment %d: %s (%p) is not %d-byte aligned", s, b.what, b.p, SDP_ALIGN);
        }
        for (size_t k = 0; k < bufs.size(); ++k) {
            const Buf &b = bufs[k];
            const MemKind kind = k < n_state ? state_kind : grad_kind;
            SDP_TRY(kind == kDeviceMem   ? check_device_ptr(ctx, b.p, b.bytes, b.what, s)
                    : kind == kPinnedHost ? check_pinned_ptr(b.p, b.bytes, b.what, s)
                                          : check_host_ptr(b.p, b.what, s));
            Range rg{(uintptr_t)b.p, (uintptr_t)b.p + b.bytes, s, b.what};
            (k < n_state ? states : grads).push_back(rg);
        }
    }
    // states pairwise disjoint; gradients disjoint from every state
    std::sort(states.begin(), states.end(), [](const Range &x, const Range &y) { return x.a < y.a; });
    for (size_t k = 1; k < states.size(); ++k)
        if (overlap(states[k - 1], states[k]))
            return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d %s overlaps segment %d %s", states[k - 1].seg,
                        states[k - 1].what, states[k].seg, states[k].what);
    for (const Range &g : grads) {
        auto it = std::upper_bound(states.begin(), states.end(), g.a,
                                   [](uintptr_t v, const Range &x) { return v < x.a; });
        if (it != states.end() && overlap(*it, g))
            return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d gradient overlaps segment %d %s", g.seg, it->seg, it->what);
        if (it != states.begin() && overlap(*(it - 1), g))
            return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d gradient overlaps segment %d %s", g.seg, (it - 1)->seg,
                        (it - 1)->what);
    }
    *R_out = R;
    return SDP_OK;
}

int check_chunk(int64_t chunk, bool allow_zero) {
    if (chunk < 0 || (chunk == 0 && !allow_zero) || chunk % SDP_NORM_TILE != 0)
        return fail(SDP_ERR_INVALID_ARGUMENT, "chunk_elems must be a %spositive multiple of %d (got %lld)",
                    allow_zero ? "zero or " : "", SDP_NORM_TILE, (long long)chunk);
    return SDP_OK;
}

// ---- workspace ----------------------------------------------------------

double *tile_partials(sdp_ctx *ctx, int64_t tile) { return ctx->partials + 2 * sdp::kNormSplit * tile; }

int ensure_partials(sdp_ctx *ctx, int64_t tiles) {
    const int64_t n = tiles * sdp::kNormSplit;
    if (n <= ctx->partials_cap) return SDP_OK;
    HIP_TRY(hipDeviceSynchronize());
    if (ctx->partials) HIP_TRY(hipFree(ctx->partials));
    ctx->partials = nullptr;
    ctx->partials_cap = 0;
    int64_t cap = std::max<int64_t>(n, 4096);
    // each span partial is a double-double pair; the finalize's first stage
    // writes one pair per kMergeRun of them after the last
    const int64_t pairs = cap + cdiv(cap, sdp::kMergeRun);
    if (hipMalloc(&ctx->partials, (size_t)pairs * 2 * sizeof(double)) != hipSuccess) {
        (void)hipGetLastError();
        ctx->partials = nullptr;
        return fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate %lld norm partials", (long long)cap);
    }
    ctx->partials_cap = cap;
    return SDP_OK;
}

int ensure_gbar(sdp_ctx *ctx, int64_t n) {
    if (n <= ctx->gbar_cap) return SDP_OK;
    HIP_TRY(hipDeviceSynchronize());
    if (ctx->gbar) HIP_TRY(hipFree(ctx->gbar));
    ctx->gbar = nullptr;
    ctx->gbar_cap = 0;
    if (hipMalloc(&ctx->gbar, (size_t)n * sizeof(float)) != hipSuccess) {
        (void)hipGetLastError();
        ctx->gbar = nullptr;
        return fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate %lld floats for the stored mean gradient", (long long)n);
    }
    ctx->gbar_cap = n;
    return SDP_OK;
}

Plan make_plan(const sdp_segment *segs, int32_t n_segs) {
    Plan p;
    for (int32_t s = 0; s < n_segs; ++s) {
        p.tile_base.push_back(p.tiles);
        p.gbar_base.push_back(p.gbar_elems);
        p.tiles += cdiv(segs[s].numel, SDP_NORM_TILE);
        p.gbar_elems += round_up(segs[s].numel, 64);  // 256-byte aligned segment bases
    }
    return p;
}

bool device_gbar(const sdp_ctx *ctx, int32_t R) {
    if (ctx->flags & SDP_FLAG_DEVICE_GBAR_ALWAYS) return true;
    if (ctx->flags & SDP_FLAG_DEVICE_GBAR_NEVER) return false;
    return R > 4;
}

// ---- timing -------------------------------------------------------------

// Timing events kept ready by sdp_ctx_set_timing: two per timed launch,
// enough for a few host-route calls of a few dozen pieces.
constexpr size_t kTimingEvents = 256;

hipEvent_t take_event(sdp_ctx *ctx) {
    if (!ctx->pool.empty()) {
        hipEvent_t e = ctx->pool.back();
        ctx->pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    return e;
}

hipEvent_t timed_begin(sdp_ctx *ctx, hipStream_t s) {
    if (!ctx->timing) return nullptr;
    hipEvent_t a = take_event(ctx);
    if (a && hipEventRecord(a, s) != hipSuccess) {
        (void)hipGetLastError();
        ctx->pool.push_back(a);
        return nullptr;
    }
    return a;
}

void timed_end(sdp_ctx *ctx, hipStream_t s, hipEvent_t a, int kind, int64_t elems) {
    if (!ctx->timing || !a) return;
    hipEvent_t b = take_event(ctx);
    if (!b || hipEventRecord(b, s) != hipSuccess) {
        (void)hipGetLastError();
        ctx->pool.push_back(a);
        if (b) ctx->pool.push_back(b);
        return;
    }
    ctx->timed.push_back({kind, a, b, elems});
}

// ---- launches shared by the modes ------------------------------------------

int norm_launch(sdp_ctx *ctx, int32_t R, const uint16_t *const *g, int64_t n, double *partials, float *gbar_out,
                hipStream_t s) {
    sdp::NormArgs a{};
    for (int32_t r = 0; r < R; ++r) a.g[r] = g[r];
    a.n = n;
    a.partials = partials;
    a.gbar_out = gbar_out;
    hipEvent_t t0 = timed_begin(ctx, s);
    HIP_TRY(sdp::launch_norm_partials(R, a, ctx->norm_store_lds_pad, s));
    timed_end(ctx, s, t0, kNorm, n);
    return SDP_OK;
}

int finalize_launch(sdp_ctx *ctx, int64_t tiles, double max_grad_norm, hipStream_t s) {
    hipEvent_t t0 = timed_begin(ctx, s);
    HIP_TRY(sdp::launch_norm_finalize(ctx->partials, tiles * sdp::kNormSplit, ctx->partials + 2 * ctx->partials_cap,
                                      max_grad_norm, ctx->ns, s));
    timed_end(ctx, s, t0, kFinalize, tiles);
    return SDP_OK;
}

void fill_consts(const sdp_adamw_params *hp, sdp::UpdateArgs &a) {
    const double t = (double)hp->step;
    const double bc1 = 1.0 - std::pow(hp->beta1, t);
    const double bc2 = 1.0 - std::pow(hp->beta2, t);
    a.lr_wd = hp->lr * hp->weight_decay;
    a.beta1 = hp->beta1;
    a.one_minus_beta1 = 1.0 - hp->beta1;
    a.beta2 = hp->beta2;
    a.one_minus_beta2 = 1.0 - hp->beta2;
    a.step_size = hp->lr / bc1;
    a.inv_bc2 = 1.0 / bc2;
    a.eps = hp->eps;
}

int update_launch(sdp_ctx *ctx, int32_t R, const sdp_adamw_params *hp, float *p, float *m, float *v, uint16_t *pb,
                  const uint16_t *const *g, const float *gbar, int64_t n, hipStream_t s) {
    sdp::UpdateArgs a{};
    a.p = p;
    a.m = m;
    a.v = v;
    a.pb = pb;
    if (!gbar)
        for (int32_t r = 0; r < R; ++r) a.g[r] = g[r];
    a.gbar = gbar;
    a.n = n;
    a.ns = ctx->ns;
    fill_consts(hp, a);
    hipEvent_t t0 = timed_begin(ctx, s);
    HIP_TRY(sdp::launch_update(R, a, ctx->update_max_blocks, ctx->update_lds_pad, s));
    timed_end(ctx, s, t0, kUpdate, n);
    return SDP_OK;
}

// Order this call's work after the previous call's (they share workspace).
int order_after_last(sdp_ctx *ctx, hipStream_t s) {
    if (ctx->last_done_valid) HIP_TRY(hipStreamWaitEvent(s, ctx->last_done, 0));
    return SDP_OK;
}

int mark_done(sdp_ctx *ctx, hipStream_t s) {
    HIP_TRY(hipEventRecord(ctx->last_done, s));
    ctx->last_done_valid = true;
    return SDP_OK;
}

namespace {
// xorshift64* (Vigna): the next draw of the context's jitter generator, as
// a number in [0, bound)
uint32_t jitter_draw(sdp_ctx *ctx, uint32_t bound) {
    uint64_t x = ctx->jitter_state;
    x ^= x >> 12;
    x ^= x << 25;
    x ^= x >> 27;
    ctx->jitter_state = x;
    return (uint32_t)(((x * 2685821657736338717ull) >> 32) % bound);
}
}  // namespace

int jitter_stream(sdp_ctx *ctx, hipStream_t s) {
    if (!(ctx->flags & SDP_FLAG_DEBUG_JITTER)) return SDP_OK;
    // s_sleep 64 is about 4,096 clocks, 1.7-1.8 us at the clocks measured:
    // up to 116 of them is up to about 200 us
    HIP_TRY(sdp::launch_sleep((int)jitter_draw(ctx, 117), s));
    return SDP_OK;
}

void jitter_host(sdp_ctx *ctx) {
    if (!(ctx->flags & SDP_FLAG_DEBUG_JITTER)) return;
    std::this_thread::sleep_for(std::chrono::microseconds(jitter_draw(ctx, 201)));
}

int read_norm(sdp_ctx *ctx, hipStream_t s, NormState *out) {
    HIP_TRY(hipMemcpyAsync(ctx->ns_host, ctx->ns, sizeof(NormState), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    *out = *ctx->ns_host;
    return SDP_OK;
}

int sync_streams(sdp_ctx *ctx) {
    HIP_TRY(hipStreamSynchronize(ctx->s_copy));
    HIP_TRY(hipStreamSynchronize(ctx->s_comp));
    return SDP_OK;
}

// ---- device mode ----------------------------------------------------------

int device_norm(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int32_t R, const Plan &plan, bool store_gbar,
                double max_grad_norm, hipStream_t s) {
    for (int32_t k = 0; k < n_segs; ++k)
        SDP_TRY(norm_launch(ctx, R, segs[k].grads, segs[k].numel, tile_partials(ctx, plan.tile_base[k]),
                            store_gbar ? ctx->gbar + plan.gbar_base[k] : nullptr, s));
    return finalize_launch(ctx, plan.tiles, max_grad_norm, s);
}

// ---- chunks and staging slots -------------------------------------------

Slot slot_at(const sdp_ctx *ctx, int k) {
    Slot sl{};
    const int64_t C = ctx->max_chunk;
    char *b = ctx->staging + (size_t)k * ctx->slot_bytes;
    sl.p = (float *)b;
    sl.m = sl.p + C;
    sl.v = sl.m + C;
    sl.pb = (uint16_t *)(sl.v + C);
    for (int r = 0; r < ctx->max_ranks; ++r) sl.g[r] = sl.pb + C + (size_t)r * C;
    return sl;
}

std::vector<Chunk> make_chunks(const sdp_segment *segs, int32_t n_segs, int64_t C) {
    std::vector<Chunk> out;
    for (int32_t s = 0; s < n_segs; ++s)
        for (int64_t off = 0; off < segs[s].numel; off += C)
            out.push_back({s, off, std::min(C, segs[s].numel - off)});
    return out;
}

size_t off_in_slot(const sdp_ctx *ctx, int sl, const void *p) {
    return (size_t)((const char *)p - (ctx->staging + (size_t)sl * ctx->slot_bytes));
}

int stream_common_checks(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int64_t chunk, bool grads_only,
                         int32_t *R) {
    if (!ctx->staging) return fail(SDP_ERR_CHUNK_TOO_LARGE, "context was created without streamed-mode staging");
    SDP_TRY(check_chunk(chunk, false));
    if (chunk > ctx->max_chunk)
        return fail(SDP_ERR_CHUNK_TOO_LARGE, "chunk_elems %lld exceeds the context's %lld", (long long)chunk,
                    (long long)ctx->max_chunk);
    const MemKind host_kind = (ctx->flags & SDP_FLAG_STREAM_STAGED) ? kAnyHost : kPinnedHost;
    SDP_TRY(validate_segments(ctx, segs, n_segs, host_kind, host_kind, grads_only, R));
    if (*R > ctx->max_ranks)
        return fail(SDP_ERR_INVALID_ARGUMENT, "n_ranks %d exceeds the context's max_ranks %d", *R, ctx->max_ranks);
    return SDP_OK;
}

// ---- host threads and pinned stage buffers ------------------------------

// Host threads of a context: SDP_STAGING_THREADS, else the hardware
// threads, at most 16 (the calling thread counts as one of them).
int default_host_threads() {
    int threads = (int)std::min(16u, std::max(1u, std::thread::hardware_concurrency()));
    if (const char *env = std::getenv("SDP_STAGING_THREADS")) threads = std::max(1, std::min(256, std::atoi(env)));
    return threads;
}

int default_staged_copy_threads() {
    int threads = kStagedCopyThreads;
    if (const char *env = std::getenv("SDP_STAGED_COPY_THREADS")) threads = std::max(1, std::min(256, std::atoi(env)));
    return threads;
}

HostPool *new_pool(const sdp_ctx *ctx, int threads) {
    return new HostPool(threads - 1, (ctx->flags & SDP_FLAG_HOST_PIN_THREADS) != 0);
}

// The host threads and the two pinned stage buffers of parameter delivery and
// the host-update route, created on first use.
int ensure_host_stage(sdp_ctx *ctx) {
    if (!ctx->copier) ctx->copier = new_pool(ctx, default_host_threads());
    if (!ctx->stage) {
        if (hipHostMalloc(&ctx->stage, 2 * stage_bytes(ctx), hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            ctx->stage = nullptr;
            return fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate %zu bytes of pinned stage buffers",
                        2 * stage_bytes(ctx));
        }
        ctx->stage_used[0] = ctx->stage_used[1] = false;
        const int rc = device_map_offset(ctx->stage, &ctx->stage_map);
        if (rc != SDP_OK) {
            (void)hipHostFree(ctx->stage);
            ctx->stage = nullptr;
            return rc;
        }
    }
    return SDP_OK;
}

int device_map_offset(const void *p, ptrdiff_t *out) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, p) != hipSuccess || at.type != hipMemoryTypeHost || !at.devicePointer) {
        (void)hipGetLastError();
        return fail(SDP_ERR_HIP, "pinned buffer %p has no device mapping", p);
    }
    *out = (const char *)at.devicePointer - (const char *)p;
    return SDP_OK;
}

bool is_pinned_host(const void *p) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return at.type == hipMemoryTypeHost;
}

}  // namespace sdprt

using namespace sdprt;

// ===========================================================================
// exported

extern "C" {

const char *sdp_status_string(int status) {
    switch (status) {
        case SDP_OK: return "SDP_OK";
        case SDP_ERR_INVALID_ARGUMENT: return "SDP_ERR_INVALID_ARGUMENT";
        case SDP_ERR_ALIGNMENT: return "SDP_ERR_ALIGNMENT";
        case SDP_ERR_NOT_DEVICE_MEMORY: return "SDP_ERR_NOT_DEVICE_MEMORY";
        case SDP_ERR_NOT_PINNED: return "SDP_ERR_NOT_PINNED";
        case SDP_ERR_CHUNK_TOO_LARGE: return "SDP_ERR_CHUNK_TOO_LARGE";
        case SDP_ERR_OUT_OF_MEMORY: return "SDP_ERR_OUT_OF_MEMORY";
        case SDP_ERR_HIP: return "SDP_ERR_HIP";
        case SDP_ERR_NONFINITE: return "SDP_ERR_NONFINITE";
        default: return "SDP_ERR_UNKNOWN";
    }
}

const char *sdp_last_error(void) { return t_err.c_str(); }

int sdp_plan(const int64_t *numels, int32_t n_segs, int64_t chunk_elems, int64_t *n_chunks_out, int64_t *n_tiles_out) {
    t_err.clear();
    if (!numels || n_segs < 1 || !n_chunks_out || !n_tiles_out)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_plan: NULL argument or no segments");
    SDP_TRY(check_chunk(chunk_elems, false));
    int64_t ch = 0, ti = 0;
    for (int32_t s = 0; s < n_segs; ++s) {
        if (numels[s] < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_plan: segment %d has numel < 1", s);
        ch += cdiv(numels[s], chunk_elems);
        ti += cdiv(numels[s], SDP_NORM_TILE);
    }
    *n_chunks_out = ch;
    *n_tiles_out = ti;
    return SDP_OK;
}

int sdp_bytes_per_elem(int streamed, int32_t n_ranks, uint32_t flags, double *hbm_or_h2d, double *d2h) {
    t_err.clear();
    if (!hbm_or_h2d || !d2h || n_ranks < 1 || n_ranks > SDP_MAX_RANKS)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_bytes_per_elem: bad argument");
    const double R = n_ranks;
    if (streamed) {
        const bool cache = !(flags & SDP_FLAG_STREAM_GBAR_NEVER);
        *hbm_or_h2d = cache ? 12.0 + 2.0 * R : 12.0 + 4.0 * R;
        *d2h = (flags & SDP_FLAG_STREAM_HOST_CAST) ? 12.0 : 14.0;
    } else {
        bool cache = (flags & SDP_FLAG_DEVICE_GBAR_ALWAYS) ? true
                     : (flags & SDP_FLAG_DEVICE_GBAR_NEVER) ? false
                                                            : (n_ranks > 4);
        // norm pass reads 2R (+ writes 4 if storing g_bar); update reads
        // 12 + (2R or 4) and writes 14
        *hbm_or_h2d = cache ? 2.0 * R + 4.0 + 4.0 + 12.0 + 14.0 : 2.0 * R + 2.0 * R + 12.0 + 14.0;
        *d2h = 0.0;
    }
    return SDP_OK;
}

}  // extern "C"

namespace {

int check_model_args(int schedule, const int64_t *numels, int32_t n_segs, int32_t n_ranks, const sdp_rates *r,
                     std::vector<int64_t> *sizes) {
    if (schedule < SDP_SCHED_STREAMED || schedule > SDP_SCHED_HOST_ROUTE_BF16)
        return fail(SDP_ERR_INVALID_ARGUMENT, "unknown schedule %d", schedule);
    if (!numels || n_segs < 1 || !r) return fail(SDP_ERR_INVALID_ARGUMENT, "NULL argument or no segments");
    if (n_ranks < 1 || n_ranks > SDP_MAX_RANKS)
        return fail(SDP_ERR_INVALID_ARGUMENT, "n_ranks must be in 1..%d", SDP_MAX_RANKS);
    const double pos[] = {r->h2d_gbs,    r->d2h_gbs,  r->both_gbs,     r->norm_gbs,
                          r->update_gbs, r->host_gbs, r->host_adam_gbs};
    const double nonneg[] = {r->copy_cmd_us, r->launch_us, r->sync_us, r->host_task_us, r->dep_us,
                             r->dma_host_cost, r->host_issue_us};
    for (double x : pos)
        if (!(std::isfinite(x) && x > 0.0)) return fail(SDP_ERR_INVALID_ARGUMENT, "rates must be finite and > 0");
    for (double x : nonneg)
        if (!(std::isfinite(x) && x >= 0.0))
            return fail(SDP_ERR_INVALID_ARGUMENT, "fixed costs must be finite and >= 0");
    sizes->assign(numels, numels + n_segs);
    for (int32_t s = 0; s < n_segs; ++s)
        if (numels[s] < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d has numel < 1", s);
    return SDP_OK;
}

sdp_sched::Rates to_rates(const sdp_rates *r) {
    return sdp_sched::Rates{r->h2d_gbs,   r->d2h_gbs,  r->both_gbs, r->copy_cmd_us,  r->norm_gbs,
                            r->update_gbs, r->launch_us, r->sync_us,  r->host_gbs,     r->host_task_us,
                            r->host_adam_gbs, r->dep_us, r->dma_host_cost, r->host_issue_us};
}

int model_chunk_ok(const std::vector<int64_t> &sizes, int64_t chunk) {
    SDP_TRY(check_chunk(chunk, false));
    int64_t n = 0;
    for (int64_t x : sizes) n += cdiv(x, chunk);
    if (n > (int64_t)1 << 22) return fail(SDP_ERR_INVALID_ARGUMENT, "%lld chunks: too many to model", (long long)n);
    return SDP_OK;
}

}  // namespace

extern "C" {

int sdp_predict_step(int schedule, const int64_t *numels, int32_t n_segs, int32_t n_ranks, int64_t chunk_elems,
                     uint32_t flags, const sdp_rates *rates, sdp_prediction *out) {
    t_err.clear();
    std::vector<int64_t> sizes;
    SDP_TRY(check_model_args(schedule, numels, n_segs, n_ranks, rates, &sizes));
    if (!out) return fail(SDP_ERR_INVALID_ARGUMENT, "out is NULL");
    SDP_TRY(model_chunk_ok(sizes, chunk_elems));
    const sdp_sched::Prediction p = sdp_sched::predict(schedule, sizes, n_ranks, chunk_elems,
                                                       !(flags & SDP_FLAG_STREAM_GBAR_NEVER),
                                                       (flags & SDP_FLAG_STREAM_HOST_CAST) != 0, to_rates(rates));
    out->predicted_ms = p.predicted_ms;
    out->bound_ms = p.bound_ms;
    out->h2d_ms = p.h2d_ms;
    out->d2h_ms = p.d2h_ms;
    out->link_ms = p.link_ms;
    out->gpu_ms = p.gpu_ms;
    out->host_ms = p.host_ms;
    out->dram_ms = p.dram_ms;
    out->n_chunks = p.n_chunks;
    return SDP_OK;
}

int sdp_tune_chunk(int schedule, const int64_t *numels, int32_t n_segs, int32_t n_ranks, uint32_t flags,
                   const sdp_rates *rates, const int64_t *candidates, int32_t n_candidates, int64_t *best_out,
                   double *predicted_ms_out) {
    t_err.clear();
    std::vector<int64_t> sizes;
    SDP_TRY(check_model_args(schedule, numels, n_segs, n_ranks, rates, &sizes));
    if (!candidates || n_candidates < 1 || !best_out)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_tune_chunk: no candidates or best_out is NULL");
    for (int32_t k = 0; k < n_candidates; ++k) SDP_TRY(model_chunk_ok(sizes, candidates[k]));
    double best = std::numeric_limits<double>::infinity();
    for (int32_t k = 0; k < n_candidates; ++k) {
        const double ms = sdp_sched::predict(schedule, sizes, n_ranks, candidates[k],
                                             !(flags & SDP_FLAG_STREAM_GBAR_NEVER),
                                             (flags & SDP_FLAG_STREAM_HOST_CAST) != 0, to_rates(rates))
                              .predicted_ms;
        if (predicted_ms_out) predicted_ms_out[k] = ms;
        if (ms < best) {
            best = ms;
            *best_out = candidates[k];
        }
    }
    return SDP_OK;
}

int sdp_host_alloc(void **out, size_t bytes) {
    t_err.clear();
    if (!out || bytes == 0) return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_host_alloc: bad argument");
    *out = nullptr;
    hipError_t e = hipHostMalloc(out, bytes, hipHostMallocDefault);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        *out = nullptr;
        return fail(SDP_ERR_OUT_OF_MEMORY, "hipHostMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    }
    return SDP_OK;
}

int sdp_host_free(void *p) {
    t_err.clear();
    if (!p) return SDP_OK;
    HIP_TRY(hipHostFree(p));
    return SDP_OK;
}

int sdp_ctx_create(sdp_ctx **out, int device, int64_t max_chunk_elems, int32_t max_ranks, uint32_t flags) {
    t_err.clear();
    if (!out) return fail(SDP_ERR_INVALID_ARGUMENT, "out is NULL");
    *out = nullptr;
    if (max_ranks < 1 || max_ranks > SDP_MAX_RANKS)
        return fail(SDP_ERR_INVALID_ARGUMENT, "max_ranks must be in 1..%d", SDP_MAX_RANKS);
    SDP_TRY(check_chunk(max_chunk_elems, true));
    const uint32_t known = SDP_FLAG_DEVICE_GBAR_NEVER | SDP_FLAG_DEVICE_GBAR_ALWAYS | SDP_FLAG_STREAM_GBAR_NEVER |
                           SDP_FLAG_DEBUG_POISON | SDP_FLAG_STREAM_STAGED | SDP_FLAG_HOST_PIN_THREADS |
                           SDP_FLAG_STREAM_HOST_CAST | SDP_FLAG_DEBUG_JITTER;
    if (flags & ~known) return fail(SDP_ERR_INVALID_ARGUMENT, "unknown context flags 0x%x", flags & ~known);
    if ((flags & SDP_FLAG_DEVICE_GBAR_NEVER) && (flags & SDP_FLAG_DEVICE_GBAR_ALWAYS))
        return fail(SDP_ERR_INVALID_ARGUMENT, "DEVICE_GBAR_NEVER and DEVICE_GBAR_ALWAYS are exclusive");
    int ndev = 0;
    HIP_TRY(hipGetDeviceCount(&ndev));
    if (device < 0 || device >= ndev) return fail(SDP_ERR_INVALID_ARGUMENT, "device %d out of range (%d GPUs)", device, ndev);
    DeviceGuard guard(device);
    sdp_ctx *c = new sdp_ctx();
    c->device = device;
    c->max_chunk = max_chunk_elems;
    c->max_ranks = max_ranks;
    c->flags = flags;
    c->jitter_state = 0x9E3779B97F4A7C15ull;
    if (const char *env = std::getenv("SDP_JITTER_SEED")) c->jitter_state ^= std::strtoull(env, nullptr, 10);
    if (c->jitter_state == 0) c->jitter_state = 1;  // xorshift's one fixed point
    if (const char *env = std::getenv("SDP_UPDATE_MAX_BLOCKS")) c->update_max_blocks = std::max(0, std::atoi(env));
    int rc = SDP_OK;
    auto bail = [&](int status) {
        sdp_ctx_destroy(c);
        return status;
    };
    {
        // residency caps: the compute unit's LDS split over the blocks that
        // may stay on it (SDP_UPDATE_BLOCKS_PER_CU and
        // SDP_NORM_STORE_BLOCKS_PER_CU override; 0 lifts a cap)
        int lds_cu = 0, lds_block = 0;
        if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device) != hipSuccess ||
            hipDeviceGetAttribute(&lds_block, hipDeviceAttributeMaxSharedMemoryPerBlock, device) != hipSuccess) {
            (void)hipGetLastError();
            return bail(fail(SDP_ERR_HIP, "cannot query the device's LDS size"));
        }
        auto pad_for = [&](const char *env_name, int per_cu, int static_lds) {
            if (const char *env = std::getenv(env_name)) per_cu = std::max(0, std::atoi(env));
            if (per_cu <= 0) return 0;
            const int pad = (lds_cu / per_cu - static_lds) / 1024 * 1024;
            return pad > 0 && pad + static_lds <= lds_block ? pad : 0;
        };
        c->update_lds_pad = pad_for("SDP_UPDATE_BLOCKS_PER_CU", sdp::kUpdateBlocksPerCU, 0);
        // the norm pass's own LDS: two 4-entry FP64 arrays for the block merge
        c->norm_store_lds_pad = pad_for("SDP_NORM_STORE_BLOCKS_PER_CU", sdp::kNormStoreBlocksPerCU, 64);
    }
#define CTX_HIP(expr)                                                                                \
    do {                                                                                             \
        hipError_t e_ = (expr);                                                                      \
        if (e_ != hipSuccess) {                                                                      \
            (void)hipGetLastError();                                                                 \
            return bail(fail(SDP_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)));           \
        }                                                                                            \
    } while (0)
    CTX_HIP(hipStreamCreateWithFlags(&c->s_copy, hipStreamNonBlocking));
    CTX_HIP(hipStreamCreateWithFlags(&c->s_comp, hipStreamNonBlocking));
    for (int k = 0; k < 2; ++k) {
        CTX_HIP(hipEventCreateWithFlags(&c->h2d_done[k], hipEventDisableTiming));
        CTX_HIP(hipEventCreateWithFlags(&c->slot_free[k], hipEventDisableTiming));
    }
    CTX_HIP(hipEventCreateWithFlags(&c->last_done, hipEventDisableTiming));
    CTX_HIP(hipEventCreateWithFlags(&c->copy_done, hipEventDisableTiming));
    if (hipMalloc(&c->ns, sizeof(NormState)) != hipSuccess) {
        (void)hipGetLastError();
        return bail(fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate the norm state"));
    }
    CTX_HIP(hipMemset(c->ns, 0, sizeof(NormState)));
    if (hipHostMalloc(&c->ns_host, sizeof(NormState), hipHostMallocDefault) != hipSuccess) {
        (void)hipGetLastError();
        return bail(fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate the pinned norm mirror"));
    }
    // pinned streamed mode with the BF16 parameters rounded on the host waits
    // on each chunk's returning copies, and then the runtime's large copies
    // ran slower than the library's kernel (183 against 144 ms per step on
    // the Qwen3-14B layer at 32M-element chunks): the kernel takes them all
    c->d2h_kernel_max = ((flags & SDP_FLAG_STREAM_HOST_CAST) && !(flags & SDP_FLAG_STREAM_STAGED))
                            ? std::numeric_limits<int64_t>::max()
                            : kD2HKernelMaxBytes;
    if (const char *env = std::getenv("SDP_D2H_KERNEL_MAX_BYTES")) c->d2h_kernel_max = std::atoll(env);
    c->d2h_kernel_blocks = 0;
    if (const char *env = std::getenv("SDP_D2H_KERNEL_BLOCKS"))
        c->d2h_kernel_blocks = std::max(1, std::min(65535, std::atoi(env)));
    if (max_chunk_elems > 0) {
        c->slot_bytes = (size_t)(14 + 2 * max_ranks) * (size_t)max_chunk_elems;
        if (hipMalloc(&c->staging, 2 * c->slot_bytes) != hipSuccess) {
            (void)hipGetLastError();
            c->staging = nullptr;
            return bail(fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate 2 x %zu bytes of staging", c->slot_bytes));
        }
    }
    if (flags & SDP_FLAG_STREAM_STAGED) {
        if (max_chunk_elems <= 0)
            return bail(fail(SDP_ERR_INVALID_ARGUMENT, "SDP_FLAG_STREAM_STAGED needs max_chunk_elems > 0"));
        const size_t out_bytes = 14 * (size_t)max_chunk_elems;
        if (hipHostMalloc(&c->bounce_in, kInBufs * c->slot_bytes, hipHostMallocDefault) != hipSuccess ||
            hipHostMalloc(&c->bounce_out, kOutBufs * out_bytes, hipHostMallocDefault) != hipSuccess) {
            (void)hipGetLastError();
            return bail(fail(SDP_ERR_OUT_OF_MEMORY, "cannot allocate %zu bytes of pinned bounce buffers",
                             kInBufs * c->slot_bytes + kOutBufs * out_bytes));
        }
        for (int k = 0; k < kInBufs; ++k)
            CTX_HIP(hipEventCreateWithFlags(&c->bin_done[k], hipEventDisableTiming));
        rc = device_map_offset(c->bounce_out, &c->bounce_out_map);
        if (rc != SDP_OK) return bail(rc);
    }
    if (flags & (SDP_FLAG_STREAM_STAGED | SDP_FLAG_STREAM_HOST_CAST)) {
        if (max_chunk_elems <= 0)
            return bail(fail(SDP_ERR_INVALID_ARGUMENT, "SDP_FLAG_STREAM_HOST_CAST needs max_chunk_elems > 0"));
        // the host threads' work on results that have landed waits for these
        for (int k = 0; k < kOutBufs; ++k)
            CTX_HIP(hipEventCreateWithFlags(&c->d2h_done[k], hipEventDisableTiming));
        c->copier = new_pool(c, default_host_threads());
        c->staged_copy_threads = default_staged_copy_threads();
    }
    rc = ensure_partials(c, 4096);
    if (rc != SDP_OK) return bail(rc);
#undef CTX_HIP
    *out = c;
    return SDP_OK;
}

void sdp_ctx_destroy(sdp_ctx *ctx) {
    if (!ctx) return;
    DeviceGuard guard(ctx->device);
    (void)hipDeviceSynchronize();
    for (const Timed &t : ctx->timed) {
        (void)hipEventDestroy(t.a);
        (void)hipEventDestroy(t.b);
    }
    for (hipEvent_t e : ctx->pool) (void)hipEventDestroy(e);
    for (int k = 0; k < 2; ++k) {
        if (ctx->h2d_done[k]) (void)hipEventDestroy(ctx->h2d_done[k]);
        if (ctx->slot_free[k]) (void)hipEventDestroy(ctx->slot_free[k]);
    }
    if (ctx->last_done) (void)hipEventDestroy(ctx->last_done);
    if (ctx->copy_done) (void)hipEventDestroy(ctx->copy_done);
    if (ctx->s_copy) (void)hipStreamDestroy(ctx->s_copy);
    if (ctx->s_comp) (void)hipStreamDestroy(ctx->s_comp);
    if (ctx->staging) (void)hipFree(ctx->staging);
    if (ctx->bounce_in) (void)hipHostFree(ctx->bounce_in);
    if (ctx->stage) (void)hipHostFree(ctx->stage);
    if (ctx->bounce_out) (void)hipHostFree(ctx->bounce_out);
    for (int k = 0; k < kInBufs; ++k)
        if (ctx->bin_done[k]) (void)hipEventDestroy(ctx->bin_done[k]);
    for (int k = 0; k < kOutBufs; ++k)
        if (ctx->d2h_done[k]) (void)hipEventDestroy(ctx->d2h_done[k]);
    delete ctx->copier;
    if (ctx->partials) (void)hipFree(ctx->partials);
    if (ctx->gbar) (void)hipFree(ctx->gbar);
    if (ctx->ns) (void)hipFree(ctx->ns);
    if (ctx->ns_host) (void)hipHostFree(ctx->ns_host);
    (void)hipGetLastError();
    delete ctx;
}

int sdp_agg_adam_step(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, const sdp_adamw_params *hp,
                      int64_t chunk_elems, void *stream, double *grad_norm_out) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    SDP_TRY(check_hparams(hp));
    SDP_TRY(check_chunk(chunk_elems, true));
    DeviceGuard guard(ctx->device);
    int32_t R = 0;
    SDP_TRY(validate_segments(ctx, segs, n_segs, kDeviceMem, kDeviceMem, false, &R));
    const Plan plan = make_plan(segs, n_segs);
    const bool store = device_gbar(ctx, R);
    SDP_TRY(ensure_partials(ctx, plan.tiles));
    if (store) SDP_TRY(ensure_gbar(ctx, plan.gbar_elems));
    hipStream_t s = (hipStream_t)stream;
    SDP_TRY(order_after_last(ctx, s));
    SDP_TRY(device_norm(ctx, segs, n_segs, R, plan, store, hp->max_grad_norm, s));
    for (int32_t k = 0; k < n_segs; ++k) {
        const sdp_segment &g = segs[k];
        SDP_TRY(update_launch(ctx, R, hp, g.master, g.exp_avg, g.exp_avg_sq, g.param_bf16, g.grads,
                              store ? ctx->gbar + plan.gbar_base[k] : nullptr, g.numel, s));
    }
    SDP_TRY(mark_done(ctx, s));
    if (grad_norm_out) {
        NormState st;
        SDP_TRY(read_norm(ctx, s, &st));
        *grad_norm_out = st.norm;
        if (st.nonfinite) return fail(SDP_ERR_NONFINITE, "gradient norm is not finite (%g); nothing was updated", st.norm);
    }
    return SDP_OK;
}

int sdp_grad_norm(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int device_resident, int64_t chunk_elems,
                  void *stream, double *norm_out) {
    t_err.clear();
    if (!ctx || !norm_out) return fail(SDP_ERR_INVALID_ARGUMENT, "context or norm_out is NULL");
    DeviceGuard guard(ctx->device);
    int32_t R = 0;
    NormState st{};
    if (device_resident) {
        SDP_TRY(validate_segments(ctx, segs, n_segs, kDeviceMem, kDeviceMem, true, &R));
        const Plan p = make_plan(segs, n_segs);
        SDP_TRY(ensure_partials(ctx, p.tiles));
        hipStream_t s = (hipStream_t)stream;
        SDP_TRY(order_after_last(ctx, s));
        SDP_TRY(device_norm(ctx, segs, n_segs, R, p, false, 0.0, s));
        SDP_TRY(mark_done(ctx, s));
        SDP_TRY(read_norm(ctx, s, &st));
    } else {
        SDP_TRY(stream_common_checks(ctx, segs, n_segs, chunk_elems, true, &R));
        const Plan p = make_plan(segs, n_segs);
        SDP_TRY(ensure_partials(ctx, p.tiles));
        const std::vector<Chunk> chunks =
            make_chunks(segs, n_segs, sdp_sched::norm_phase_chunk(chunk_elems, R, staged(ctx)));
        SDP_TRY(order_after_last(ctx, ctx->s_copy));
        SDP_TRY(order_after_last(ctx, ctx->s_comp));
        bool used[2] = {false, false};
        int rc = stream_norm_phase(ctx, segs, n_segs, R, p, chunks, false, 0.0, used);
        if (rc == SDP_OK) rc = read_norm(ctx, ctx->s_comp, &st);
        int rc2 = sync_streams(ctx);
        if (rc != SDP_OK) return rc;
        if (rc2 != SDP_OK) return rc2;
        SDP_TRY(mark_done(ctx, ctx->s_comp));
    }
    *norm_out = st.norm;
    if (st.nonfinite) return fail(SDP_ERR_NONFINITE, "gradient norm is not finite (%g)", st.norm);
    return SDP_OK;
}

int sdp_ctx_last_norm(sdp_ctx *ctx, double *norm, double *clip_coef, int *nonfinite) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    DeviceGuard guard(ctx->device);
    if (ctx->last_done_valid) HIP_TRY(hipEventSynchronize(ctx->last_done));
    NormState st{};
    HIP_TRY(hipMemcpy(&st, ctx->ns, sizeof st, hipMemcpyDeviceToHost));
    if (norm) *norm = st.norm;
    if (clip_coef) *clip_coef = st.clip;
    if (nonfinite) *nonfinite = st.nonfinite;
    return SDP_OK;
}

int sdp_cast_bf16(sdp_ctx *ctx, const float *src, uint16_t *dst, int64_t n, void *stream) {
    t_err.clear();
    if (!ctx || !src || !dst || n < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_cast_bf16: bad argument");
    if (!aligned(src) || !aligned(dst)) return fail(SDP_ERR_ALIGNMENT, "sdp_cast_bf16: pointers must be 16-byte aligned");
    DeviceGuard guard(ctx->device);
    SDP_TRY(check_device_ptr(ctx, src, (size_t)n * 4, "src", 0));
    SDP_TRY(check_device_ptr(ctx, dst, (size_t)n * 2, "dst", 0));
    uintptr_t a0 = (uintptr_t)src, a1 = a0 + (size_t)n * 4, b0 = (uintptr_t)dst, b1 = b0 + (size_t)n * 2;
    if (a0 < b1 && b0 < a1) return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_cast_bf16: src and dst overlap");
    HIP_TRY(sdp::launch_cast_bf16(src, dst, n, (hipStream_t)stream));
    return SDP_OK;
}

int sdp_ctx_set_timing(sdp_ctx *ctx, int enable) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    DeviceGuard guard(ctx->device);
    if (enable) {
        for (const Timed &t : ctx->timed) {
            (void)hipEventSynchronize(t.b);
            ctx->pool.push_back(t.a);
            ctx->pool.push_back(t.b);
        }
        ctx->timed.clear();
        ctx->host_adam_ms = ctx->host_wait_ms = ctx->host_issue_ms = 0.0;
        ctx->host_adam_elems = ctx->host_issues = 0;
        // events ready in advance: creating one takes host time, which a call
        // on the host-bound route would otherwise spend before its launches
        while (ctx->pool.size() < kTimingEvents) {
            hipEvent_t e = nullptr;
            HIP_TRY(hipEventCreate(&e));
            ctx->pool.push_back(e);
        }
    }
    ctx->timing = enable != 0;
    return SDP_OK;
}

int sdp_ctx_get_timing(sdp_ctx *ctx, sdp_kernel_times *out) {
    t_err.clear();
    if (!ctx || !out) return fail(SDP_ERR_INVALID_ARGUMENT, "context or out is NULL");
    DeviceGuard guard(ctx->device);
    sdp_kernel_times r{};
    for (const Timed &t : ctx->timed) {
        HIP_TRY(hipEventSynchronize(t.b));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, t.a, t.b));
        if (t.kind == kNorm) {
            r.norm_ms += ms;
            r.norm_launches++;
        } else if (t.kind == kFinalize) {
            r.finalize_ms += ms;
            r.finalize_launches++;
        } else if (t.kind == kGbar) {
            r.gbar_ms += ms;
            r.gbar_launches++;
        } else {
            r.update_ms += ms;
            r.update_launches++;
            r.update_elems += t.elems;
        }
    }
    r.host_adam_ms = ctx->host_adam_ms;
    r.host_wait_ms = ctx->host_wait_ms;
    r.host_adam_elems = ctx->host_adam_elems;
    r.host_issue_ms = ctx->host_issue_ms;
    r.host_issues = ctx->host_issues;
    *out = r;
    return SDP_OK;
}

int sdp_probe_copy(sdp_ctx *ctx, void *dst, const void *src, int64_t bytes, void *stream) {
    t_err.clear();
    if (!ctx || !dst || !src || bytes < 16 || bytes % 16 != 0)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_probe_copy: bad argument (bytes must be a positive multiple of 16)");
    if (!aligned(dst) || !aligned(src)) return fail(SDP_ERR_ALIGNMENT, "sdp_probe_copy: pointers must be 16-byte aligned");
    DeviceGuard guard(ctx->device);
    SDP_TRY(check_device_ptr(ctx, dst, (size_t)bytes, "dst", 0));
    SDP_TRY(check_device_ptr(ctx, src, (size_t)bytes, "src", 0));
    HIP_TRY(sdp::launch_copy16(dst, src, bytes / 16, ctx->update_max_blocks, (hipStream_t)stream));
    return SDP_OK;
}

int sdp_probe_memcpy(sdp_ctx *ctx, void *dst, const void *src, int64_t bytes, void *stream) {
    t_err.clear();
    if (!ctx || !dst || !src || bytes < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_probe_memcpy: bad argument");
    DeviceGuard guard(ctx->device);
    SDP_TRY(check_device_ptr(ctx, dst, (size_t)bytes, "dst", 0));
    SDP_TRY(check_device_ptr(ctx, src, (size_t)bytes, "src", 0));
    const uintptr_t a = (uintptr_t)dst, b = (uintptr_t)src;
    if (a < b + (size_t)bytes && b < a + (size_t)bytes)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_probe_memcpy: dst and src overlap");
    HIP_TRY(hipMemcpyAsync(dst, src, (size_t)bytes, hipMemcpyDeviceToDevice, (hipStream_t)stream));
    return SDP_OK;
}

int sdp_probe_update_pattern(sdp_ctx *ctx, const sdp_segment *seg, void *stream) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    DeviceGuard guard(ctx->device);
    int32_t R = 0;
    SDP_TRY(validate_segments(ctx, seg, 1, kDeviceMem, kDeviceMem, false, &R));
    sdp::UpdateArgs a{};
    a.p = seg->master;
    a.m = seg->exp_avg;
    a.v = seg->exp_avg_sq;
    a.pb = seg->param_bf16;
    for (int32_t r = 0; r < R; ++r) a.g[r] = seg->grads[r];
    a.n = seg->numel;
    hipStream_t s = (hipStream_t)stream;
    if (device_gbar(ctx, R)) {
        // the update as device mode runs it here: from stored g_bar (the
        // context's workspace; its contents do not matter to the pattern)
        SDP_TRY(ensure_gbar(ctx, seg->numel));
        SDP_TRY(order_after_last(ctx, s));
        a.gbar = ctx->gbar;
    }
    HIP_TRY(sdp::launch_update_pattern(R, a, ctx->update_lds_pad, s));
    if (a.gbar) SDP_TRY(mark_done(ctx, s));
    return SDP_OK;
}

int sdp_probe_norm_pattern(sdp_ctx *ctx, const sdp_segment *seg, void *stream) {
    t_err.clear();
    if (!ctx) return fail(SDP_ERR_INVALID_ARGUMENT, "context is NULL");
    DeviceGuard guard(ctx->device);
    int32_t R = 0;
    SDP_TRY(validate_segments(ctx, seg, 1, kDeviceMem, kDeviceMem, false, &R));
    const int64_t tiles = cdiv(seg->numel, SDP_NORM_TILE);
    SDP_TRY(ensure_partials(ctx, tiles));
    SDP_TRY(ensure_gbar(ctx, seg->numel));
    hipStream_t s = (hipStream_t)stream;
    SDP_TRY(order_after_last(ctx, s));
    sdp::NormArgs a{};
    for (int32_t r = 0; r < R; ++r) a.g[r] = seg->grads[r];
    a.n = seg->numel;
    a.partials = ctx->partials;
    a.gbar_out = ctx->gbar;
    HIP_TRY(sdp::launch_norm_pattern(R, a, ctx->norm_store_lds_pad, s));
    SDP_TRY(mark_done(ctx, s));
    return SDP_OK;
}

}  // extern "C"

namespace {

// Both link probes: H2D as runtime copies on the copy stream; D2H as runtime
// copies, or (kernel_d2h) as the streamed engine's copy kernel, one launch of
// kD2HLaunchBlocks blocks per piece storing straight into the pinned memory,
// on the compute stream.
int probe_link(sdp_ctx *ctx, void *host_a, void *host_b, void *dev_a, void *dev_b, int64_t bytes, int64_t chunk_bytes,
               int32_t reps, bool kernel_d2h, double *gbs_out, const char *name) {
    if (!ctx || !host_a || !host_b || !dev_a || !dev_b || !gbs_out || bytes < 1 || chunk_bytes < 1 || reps < 1)
        return fail(SDP_ERR_INVALID_ARGUMENT, "%s: bad argument", name);
    DeviceGuard guard(ctx->device);
    SDP_TRY(check_pinned_ptr(host_a, (size_t)bytes, "host_a", 0));
    SDP_TRY(check_pinned_ptr(host_b, (size_t)bytes, "host_b", 0));
    SDP_TRY(check_device_ptr(ctx, dev_a, (size_t)bytes, "dev_a", 0));
    SDP_TRY(check_device_ptr(ctx, dev_b, (size_t)bytes, "dev_b", 0));
    char *mapped_b = nullptr;
    if (kernel_d2h) {
        hipPointerAttribute_t at;
        if (hipPointerGetAttributes(&at, host_b) != hipSuccess || !at.devicePointer) {
            (void)hipGetLastError();
            return fail(SDP_ERR_NOT_PINNED, "%s: host_b has no device mapping", name);
        }
        mapped_b = (char *)at.devicePointer;
        if (((uintptr_t)mapped_b | (uintptr_t)dev_b | (uintptr_t)chunk_bytes) % 16 != 0)
            return fail(SDP_ERR_ALIGNMENT, "%s: buffers and chunk_bytes must be 16-byte aligned", name);
    }
    HIP_TRY(hipDeviceSynchronize());
    // Each pattern is timed on the host from its first enqueue to the end of
    // both streams, with nothing else in flight; the two directions are
    // issued chunk by chunk, interleaved, as the streamed engine issues them.
    auto copy = [&](bool h2d, int64_t off) -> hipError_t {
        const size_t len = (size_t)std::min(chunk_bytes, bytes - off);
        if (h2d)
            return hipMemcpyAsync((char *)dev_a + off, (const char *)host_a + off, len, hipMemcpyHostToDevice,
                                  ctx->s_copy);
        if (!kernel_d2h)
            return hipMemcpyAsync((char *)host_b + off, (const char *)dev_b + off, len, hipMemcpyDeviceToHost,
                                  ctx->s_comp);
        sdp::CopyBatch b{};
        b.n = 1;
        b.dst[0] = mapped_b + off;
        b.src[0] = (const char *)dev_b + off;
        b.bytes[0] = (int64_t)len;
        const int per_copy = ctx->d2h_kernel_blocks > 0 ? ctx->d2h_kernel_blocks : kD2HLaunchBlocks;
        return sdp::launch_copy_batch(b, per_copy, ctx->s_comp);
    };
    auto run = [&](bool do_h2d, bool do_d2h, double *seconds) -> hipError_t {
        const auto t0 = std::chrono::steady_clock::now();
        for (int32_t k = 0; k < reps; ++k)
            for (int64_t off = 0; off < bytes; off += chunk_bytes) {
                hipError_t e = hipSuccess;
                if (do_h2d && (e = copy(true, off)) != hipSuccess) return e;
                if (do_d2h && (e = copy(false, off)) != hipSuccess) return e;
            }
        hipError_t e = hipStreamSynchronize(ctx->s_copy);
        if (e == hipSuccess) e = hipStreamSynchronize(ctx->s_comp);
        *seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
        return e;
    };
    const double total = (double)bytes * reps;
    double sec = 0.0;
    HIP_TRY(run(true, false, &sec));
    gbs_out[0] = total / sec / 1e9;
    HIP_TRY(run(false, true, &sec));
    gbs_out[1] = total / sec / 1e9;
    HIP_TRY(run(true, true, &sec));
    gbs_out[2] = 2.0 * total / sec / 1e9;
    return SDP_OK;
}

}  // namespace

extern "C" {

int sdp_probe_link(sdp_ctx *ctx, void *host_a, void *host_b, void *dev_a, void *dev_b, int64_t bytes,
                   int64_t chunk_bytes, int32_t reps, double *gbs_out) {
    t_err.clear();
    return probe_link(ctx, host_a, host_b, dev_a, dev_b, bytes, chunk_bytes, reps, false, gbs_out, "sdp_probe_link");
}

int sdp_probe_link_kernel(sdp_ctx *ctx, void *host_a, void *host_b, void *dev_a, void *dev_b, int64_t bytes,
                          int64_t chunk_bytes, int32_t reps, double *gbs_out) {
    t_err.clear();
    return probe_link(ctx, host_a, host_b, dev_a, dev_b, bytes, chunk_bytes, reps, true, gbs_out,
                      "sdp_probe_link_kernel");
}

int sdp_probe_host_copy(sdp_ctx *ctx, void *dst, const void *src, int64_t bytes, int32_t reps, double *gbs_out) {
    t_err.clear();
    if (!ctx || !dst || !src || bytes < 1 || reps < 1 || !gbs_out)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_probe_host_copy: bad argument");
    const uintptr_t a = (uintptr_t)dst, b = (uintptr_t)src;
    if (a < b + (size_t)bytes && b < a + (size_t)bytes)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_probe_host_copy: dst and src overlap");
    if (!ctx->copier) ctx->copier = new_pool(ctx, default_host_threads());
    const Clock::time_point t0 = Clock::now();
    for (int32_t r = 0; r < reps; ++r) pool_jobs(ctx->copier, {{dst, src, (size_t)bytes}});
    const double s = ms_between(t0, Clock::now()) / 1e3;
    *gbs_out = 2.0 * (double)bytes * reps / s / 1e9;
    return SDP_OK;
}

}  // extern "C"
