/*
 * sdp.h -- C ABI of libsdp, the MI355X (gfx950) library for the data-parallel
 * optimizer update of SlideDP (arxiv 2609.34162): aggregate the BF16
 * gradients of R data-parallel ranks, clip by the global L2 norm, apply
 * mixed-precision AdamW to FP32 master weights and moments, and re-emit BF16
 * parameters.
 *
 * The paper keeps one FP32 master copy and two FP32 Adam moments per layer,
 * updated once per iteration from the gradient averaged over all ranks, and
 * hands BF16 copies of the weights to the ranks for the next forward pass
 * (Background, training-state table; Design, shared host state and
 * communication routes; Design, cross-rank pipelining and chunked overlap).
 * The paper runs that update on host CPUs.  This library runs it on the GPU,
 * either on states in device memory (sdp_agg_adam_step) or on states in
 * pinned host memory streamed through the GPU in double-buffered chunks
 * (sdp_stream_step); and, as the paper does, on host cores fed by the
 * GPU-averaged gradient (sdp_host_update_step).
 *
 * Conventions for every call:
 *  - Return value: SDP_OK (0) or a negative SDP_ERR_* status.  A failing call
 *    validates before it enqueues anything, so it has no side effects, except
 *    SDP_ERR_HIP, which reports a HIP runtime failure (text in
 *    sdp_last_error()).
 *  - sdp_last_error() returns the detail of the last failure on the calling
 *    thread (thread-local, valid until the next call on that thread).
 *  - A "stream" argument is a hipStream_t passed as void*; NULL is the null
 *    stream.  The header needs no HIP include.
 *  - The caller owns every state and gradient buffer.  The library never
 *    frees them and keeps no pointer to them after the work it enqueued
 *    completes.  The context owns its workspace.
 *  - One context is not thread-safe; different contexts are independent.
 *
 * Numerics (the paper never states the optimizer formulas; these follow
 * AdamW with decoupled decay, Loshchilov & Hutter, and Kingma & Ba bias
 * correction):
 *    g_bar[i] = fp32( (exact sum over r of bf16 G_r[i]) / R ), rounded once
 *               (an exactly zero sum gives +0; a NaN or infinite G_r[i] gives
 *               the IEEE result of the FP64 sum in rank order divided by R)
 *    norm     = sqrt( sum over all elements of all segments of g_bar^2 ) (FP64)
 *    c        = min(1, max_grad_norm / (norm + 1e-6)) if max_grad_norm > 0, else 1
 *    g        = g_bar * c
 *    p1 = p - lr*wd*p ; m' = b1*m + (1-b1)*g ; v' = b2*v + (1-b2)*g^2
 *    p' = p1 - (lr / (1 - b1^t)) * m' / (sqrt(v' / (1 - b2^t)) + eps)
 *    master = fp32(p'), exp_avg = fp32(m'), exp_avg_sq = fp32(v'),
 *    param_bf16 = bf16_rne(master)
 *  The per-element update is evaluated in FP64 registers and rounded once.
 *  The host-update route with SDP_GBAR_BF16 uses g = bf16_rne(g_bar) * c
 *  (the norm and c still come from the FP32 g_bar).
 *  A non-finite norm leaves every state and parameter unchanged.
 *  Results do not depend on the chunk size, on the mode (device or
 *  streamed) or on run-to-run scheduling: the norm is a fixed-order tree
 *  over fixed 4,096-element spans of each segment (sixteen per
 *  65,536-element tile, and chunks are whole tiles).  The host-update route
 *  with SDP_GBAR_F32 gives the same norm bits; its host cores evaluate the
 *  same FP64 expression, so its states agree with the other modes up to the
 *  last FP64 rounding before the FP32 one.
 */
#ifndef SDP_H
#define SDP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Every entry point below is exported from libsdp.so; nothing else is. */
#define SDP_API __attribute__((visibility("default")))

/* ---- status codes ------------------------------------------------------ */
#define SDP_OK 0
#define SDP_ERR_INVALID_ARGUMENT (-1)  /* NULL pointer, bad size, R out of range, aliasing */
#define SDP_ERR_ALIGNMENT (-2)         /* a buffer is not 16-byte aligned */
#define SDP_ERR_NOT_DEVICE_MEMORY (-3) /* device mode got a pointer that is not device memory of ctx's GPU, or a range that overruns its allocation */
#define SDP_ERR_NOT_PINNED (-4)        /* streamed mode got host memory that is not pinned */
#define SDP_ERR_CHUNK_TOO_LARGE (-5)   /* chunk_elems exceeds the context's staging */
#define SDP_ERR_OUT_OF_MEMORY (-6)     /* workspace allocation failed */
#define SDP_ERR_HIP (-7)               /* HIP runtime error; see sdp_last_error() */
#define SDP_ERR_NONFINITE (-8)         /* gradient norm is NaN or Inf; nothing was updated */

/* ---- constants --------------------------------------------------------- */
#define SDP_NORM_TILE 65536 /* norm tile: the norm sums in a grid fixed per tile (sixteen partials each); chunk sizes are multiples of it */
#define SDP_MAX_RANKS 16    /* largest R */
#define SDP_ALIGN 16        /* byte alignment required of every buffer */

/* ---- context flags ----------------------------------------------------- */
/* Device mode: whether the norm pass stores g_bar (4 B/element of workspace)
 * so that the update pass reads 4 B instead of 2R B per element.  Default
 * (neither flag): stored when R > 4, where it moves fewer bytes. */
#define SDP_FLAG_DEVICE_GBAR_NEVER 0x1u
#define SDP_FLAG_DEVICE_GBAR_ALWAYS 0x2u
/* Streamed mode: by default g_bar is kept in device memory between the norm
 * pass and the update pass, so each gradient crosses the host link once.
 * With this flag the gradients are streamed a second time instead. */
#define SDP_FLAG_STREAM_GBAR_NEVER 0x4u
/* Streamed mode: after each staging slot is released, fill it with a NaN
 * pattern (debug aid: a missing wait then shows up as corrupted results). */
#define SDP_FLAG_DEBUG_POISON 0x8u
/* Streamed mode, staged: the host buffers may be ordinary (pageable) memory.
 * Each chunk moves through context-owned pinned bounce buffers: host threads
 * copy chunks in ahead of their DMA (up to two chunks ahead in the update
 * pass), and copy each chunk's results out as soon as they have landed.  For
 * host states larger than the pinned memory the system grants.  Needs
 * max_chunk_elems > 0; pins 3 * (28 + 2 * max_ranks) * max_chunk_elems bytes
 * (three incoming bounce buffers shaped like a slot, three outgoing ones of
 * 14 bytes per element); host threads: SDP_STAGING_THREADS, default up to
 * 16, of which SDP_STAGED_COPY_THREADS (default 4) copy while transfers are
 * in flight in both directions.  Create such a context before allocating a
 * large host state: on the MI355X hosts measured, bounce buffers pinned
 * after 266 GB of host allocations made the update pass twice as slow. */
#define SDP_FLAG_STREAM_STAGED 0x10u
/* Host threads: keep each of the context's worker threads on one CPU of the
 * process's affinity set (the calling thread is left alone). */
#define SDP_FLAG_HOST_PIN_THREADS 0x20u
/* Streamed mode: the BF16 parameters do not cross the link.  Once a chunk's
 * FP32 master has landed in host memory, host threads round it to BF16 into
 * param_bf16 (round to nearest even, the device's bits), as the paper's host
 * rounds FP32 weights to BF16 (Design, chunked overlap).  The update pass
 * then moves 12 bytes per element each way instead of 12 in and 14 out.
 * Needs max_chunk_elems > 0; host threads as for SDP_FLAG_STREAM_STAGED.
 * Without SDP_FLAG_STREAM_STAGED every device-to-host copy then runs as the
 * library's copy kernel (SDP_D2H_KERNEL_MAX_BYTES overrides).  Combined with
 * SDP_FLAG_STREAM_STAGED it is correct but measured slower. */
#define SDP_FLAG_STREAM_HOST_CAST 0x40u
/* Debug aid for the streamed mode, the host-update route and parameter
 * delivery: before each of their copies and kernels the engines enqueue, on
 * that stream, a one-wave kernel that sleeps a random 0-200 us, and the
 * calling thread sleeps a random 0-200 us before each of its waits, host
 * copies and host updates.  It shifts the timing between the copy stream,
 * the compute stream and the host, so that a missing wait shows up (with
 * SDP_FLAG_DEBUG_POISON) as wrong results; results are unchanged otherwise.
 * The delays come from a per-context generator seeded by SDP_JITTER_SEED
 * (an unsigned integer; a fixed seed by default). */
#define SDP_FLAG_DEBUG_JITTER 0x80u

/* ---- types ------------------------------------------------------------- */
typedef struct sdp_ctx sdp_ctx;

/* Hyperparameters of one step.  step = t >= 1 is the 1-based optimizer step
 * used for bias correction; max_grad_norm <= 0 disables clipping. */
typedef struct {
    double lr, beta1, beta2, eps, weight_decay, max_grad_norm;
    int64_t step;
} sdp_adamw_params;

/* One flat layer state: all its tensors concatenated, numel elements.
 * master / exp_avg / exp_avg_sq: FP32, updated in place.
 * param_bf16: BF16 bit patterns (uint16), written.
 * grads: array of n_ranks pointers, each to numel BF16 bit patterns (read only).
 * n_ranks must be the same for every segment of a call, 1..SDP_MAX_RANKS.
 * Gradients must not overlap any state; param_bf16 must not overlap master.
 * Every pointer must be SDP_ALIGN-byte aligned; numel >= 1, any value. */
typedef struct {
    float *master;
    float *exp_avg;
    float *exp_avg_sq;
    uint16_t *param_bf16;
    const uint16_t *const *grads;
    int32_t n_ranks;
    int64_t numel;
} sdp_segment;

/* Accumulated kernel times of a context, from HIP events recorded around
 * each launch on the stream the launch uses (only while timing is on). */
typedef struct {
    double norm_ms;       /* norm-partials kernel (first pass over the gradients) */
    double finalize_ms;   /* norm finalize (both of its kernels, one launch each) */
    double update_ms;     /* fused aggregate + clip + AdamW + BF16 kernel */
    int64_t norm_launches, finalize_launches, update_launches;
    int64_t update_elems; /* elements processed by the timed update launches */
    /* host-update route (sdp_host_update_step) */
    double gbar_ms;       /* mean-gradient kernel (HIP events) */
    int64_t gbar_launches;
    double host_adam_ms;  /* host threads running AdamW (host clock) */
    double host_wait_ms;  /* host waiting for a chunk's g_bar copy to land (host clock) */
    int64_t host_adam_elems;
    double host_issue_ms; /* the calling thread enqueueing the next piece's kernel and copy (host clock) */
    int64_t host_issues;  /* pieces so enqueued */
} sdp_kernel_times;

/* ---- context ----------------------------------------------------------- */

/* Create a context on GPU `device`.  max_chunk_elems > 0 reserves two
 * streamed-mode staging slots of (14 + 2*max_ranks) * max_chunk_elems bytes
 * each (0: device mode only); it must be a multiple of SDP_NORM_TILE.
 * max_ranks in 1..SDP_MAX_RANKS bounds R for streamed mode staging.  The
 * context creates two streams (default priority) and its events.  Other
 * workspace (norm partials, cached g_bar) grows on demand.  The fused update
 * keeps at most 10 of its one-wave blocks on a compute unit, and the norm
 * pass that stores g_bar at most 4 of its blocks, through dynamic LDS that
 * they do not use; the environment variables SDP_UPDATE_BLOCKS_PER_CU and
 * SDP_NORM_STORE_BLOCKS_PER_CU, read here, set other caps (0: none). */
SDP_API int sdp_ctx_create(sdp_ctx **out, int device, int64_t max_chunk_elems,
                   int32_t max_ranks, uint32_t flags);
SDP_API void sdp_ctx_destroy(sdp_ctx *ctx);

/* ---- the update -------------------------------------------------------- */

/* Device mode: the update of each layer's FP32 master and moments from the
 * gradient averaged over the R ranks, which the paper's rank-0 worker makes
 * once per iteration on the host (Design, shared host state and
 * communication routes: the update worker and gradient return by GPU
 * reduction), here on the GPU with the states in HBM; the global-norm clip
 * before it has no counterpart in the paper.  All state and gradient buffers
 * are device memory of ctx's GPU.  Enqueues on `stream`: the norm pass over every tile of every segment
 * (segment order, then tile order), the norm finalize (a fixed-order merge of
 * the span partials, in two stages above 2,048 of them), and the
 * fused update over every element; the update reads the clip coefficient and
 * the non-finite flag from device memory, so nothing returns to the host.
 * chunk_elems (0 or a multiple of SDP_NORM_TILE) names the unit the caller
 * works in; results never depend on it, and each segment is covered by one
 * launch per kernel.  Asynchronous unless grad_norm_out is non-NULL: then the
 * call waits for the stream, stores the pre-clip norm, and returns
 * SDP_ERR_NONFINITE if it is not finite (states unchanged).  Without
 * grad_norm_out a non-finite norm still leaves the states unchanged, and
 * sdp_ctx_last_norm() reports it after the stream has finished.  The caller
 * keeps the buffers alive until the stream has finished the work. */
SDP_API int sdp_agg_adam_step(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs,
                      const sdp_adamw_params *hp, int64_t chunk_elems,
                      void *stream, double *grad_norm_out);

/* Device mode for callers that cannot allocate: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  As
 * sdp_agg_adam_step on the GPU current to the calling thread, with no
 * context: the norm partials, the finalize's merge stage and the norm state
 * live in a static device array of the library (4 MiB on each GPU it runs
 * on, held until the process ends; its address on a GPU is looked up on the
 * first call there).  The call allocates nothing, host or device.  The mean
 * gradient is not stored: the update reads the R gradient buffers again.
 * Limits: at most SDP_NOALLOC_MAX_SEGMENTS segments and SDP_NOALLOC_MAX_TILES
 * norm tiles in all (sum of ceil(numel / SDP_NORM_TILE), up to 2^30
 * elements); larger calls are rejected with SDP_ERR_INVALID_ARGUMENT before
 * anything else is checked.  Every call on a GPU uses that GPU's one array:
 * calls that overlap on one GPU (other streams, other threads) race, calls
 * on one stream are ordered.  Asynchronous on `stream` unless grad_norm_out
 * is non-NULL (then it waits and reports the norm, and SDP_ERR_NONFINITE
 * for a non-finite one, states unchanged).  Results equal sdp_agg_adam_step's
 * bit for bit. */
#define SDP_NOALLOC_MAX_SEGMENTS 64
#define SDP_NOALLOC_MAX_TILES 16384
SDP_API int sdp_agg_adam_step_noalloc(const sdp_segment *segs, int32_t n_segs, const sdp_adamw_params *hp,
                                      void *stream, double *grad_norm_out);

/* Streamed mode: the same update with the states in host memory, as the
 * paper keeps them, moved through the GPU in chunks whose transfers overlap
 * the previous chunk's work, a staging buffer being refilled only after its
 * previous consumer has finished (Design, cross-rank pipelining and chunked
 * overlap within a layer; completion and buffer reuse).  All state and
 * gradient buffers are pinned host memory
 * (e.g. from sdp_host_alloc), or any host memory when the context was
 * created with SDP_FLAG_STREAM_STAGED.  chunk_elems: a multiple of SDP_NORM_TILE,
 * at most the context's max_chunk_elems, and n_ranks <= its max_ranks.
 * Phase 1 copies each chunk's R gradients host-to-device on the copy
 * stream and runs the norm pass on the compute stream, alternating two
 * staging slots ordered by events; then the norm is finalized and read back.
 * From pinned memory its chunks fill a slot: the largest multiple of
 * SDP_NORM_TILE whose R BF16 arrays fit in (14 + 2R) * chunk_elems bytes
 * (staged, chunk_elems).
 * Phase 2 copies master/m/v of each chunk in, runs the fused update, and
 * copies master/m/v and the BF16 parameters back to the same host locations
 * on the compute stream, again double-buffered.  Device-to-host copies of up
 * to 64 MiB (all of them with SDP_FLAG_STREAM_HOST_CAST and pinned memory;
 * SDP_D2H_KERNEL_MAX_BYTES, read at context creation, overrides; 0: none)
 * run as one launch of the library's copy kernel per chunk, which stores
 * into the pinned host memory directly; larger ones are runtime copies.
 * Blocks until every copy has landed.  Returns SDP_ERR_NONFINITE (states
 * unchanged) for a non-finite norm.  grad_norm_out may be NULL. */
SDP_API int sdp_stream_step(sdp_ctx *ctx, const sdp_segment *host_segs, int32_t n_segs,
                    const sdp_adamw_params *hp, int64_t chunk_elems,
                    double *grad_norm_out);

/* Gradient formats of the host-update route: the mean gradient crosses the
 * link as FP32 (4 B/element) or rounded to BF16 (2 B/element). */
#define SDP_GBAR_F32 0
#define SDP_GBAR_BF16 1

/* Host-update route: the paper's own datapath on one GPU (Design, gradient
 * return by GPU reduction; cross-rank pipelining, the per-layer chain of
 * reduction, chunked D2H and host Adam).  The R rank gradients are device
 * memory of ctx's GPU; master/exp_avg/exp_avg_sq/param_bf16 are host memory
 * (pinned or pageable; the host threads touch them, no DMA does).
 * Phase 1 runs the norm pass and finalize over the device gradients and
 * reads the norm back.  Phase 2 walks each segment in pieces of at most
 * chunk_elems elements; at the call's start the pieces grow from
 * chunk_elems/16 by 6/5 per piece, in whole SDP_NORM_TILEs (no growth when
 * chunk_elems/16 is less than SDP_NORM_TILE): the GPU writes the piece's mean gradient into a device
 * staging slot, the copy stream moves it into a pinned stage buffer, and
 * the context's host threads run AdamW on the previous piece meanwhile
 * (double-buffered).  gbar_format SDP_GBAR_BF16
 * rounds the mean gradient to BF16 before the copy, as the paper returns
 * one BF16 gradient; the update then uses bf16(g_bar) * c, while the norm
 * and c still come from the FP32 mean.  SDP_GBAR_F32 gives the same results
 * as the other modes, up to FP64 rounding.  chunk_elems as for
 * sdp_stream_step (the context needs staging).  Blocks until every state is
 * written; returns SDP_ERR_NONFINITE (states unchanged) for a non-finite
 * norm.  grad_norm_out may be NULL.  Host threads: sdp_ctx_set_host_threads,
 * else SDP_STAGING_THREADS, else up to 16.  The first call creates them and
 * the two pinned stage buffers if the context has none. */
SDP_API int sdp_host_update_step(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs,
                         const sdp_adamw_params *hp, int64_t chunk_elems, int gbar_format,
                         double *grad_norm_out);

/* The host AdamW lane of the route on its own, for n elements of host memory:
 * master/exp_avg/exp_avg_sq updated in place and param_bf16 written from
 * gbar (FP32 or BF16 per gbar_format) and the clip coefficient clip_coef
 * (finite, >= 0), with the per-element arithmetic of the fused update (FP64,
 * no fused multiply-add, one rounding to FP32).  AVX-512 where the CPU has
 * it (SDP_HOST_SIMD=0 forces the scalar path; both give the same bits).
 * ctx may be NULL: the calling thread does the work and no GPU is needed;
 * else the context's host threads share it.  Buffers 16-byte aligned and
 * pairwise disjoint. */
SDP_API int sdp_host_adamw(sdp_ctx *ctx, float *master, float *exp_avg, float *exp_avg_sq,
                   uint16_t *param_bf16, const void *gbar, int gbar_format, int64_t n,
                   double clip_coef, const sdp_adamw_params *hp);

/* Host threads of a context (the calling thread counts as one): they run the
 * staged mode's bounce copies, the host BF16 cast and the host AdamW.
 * threads in 1..256; replaces the context's thread pool. */
SDP_API int sdp_ctx_set_host_threads(sdp_ctx *ctx, int32_t threads);
SDP_API int sdp_ctx_host_threads(sdp_ctx *ctx, int32_t *threads_out);

/* The global norm of the mean gradient alone: the L2 norm, over every
 * element of every segment of the call, of the gradient averaged over the
 * ranks (Design, gradient return by GPU reduction); the paper never clips,
 * and this is the quantity the update clips by (the first pass and finalize of
 * either mode; device_resident selects device or pinned-host buffers; only
 * grads, n_ranks and numel of each segment are read).  Blocks; chunk_elems
 * is used in streamed mode only, where the pass runs in chunks as phase 1 of
 * sdp_stream_step does.  Stores the norm even if it is not finite
 * and then returns SDP_ERR_NONFINITE. */
SDP_API int sdp_grad_norm(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs,
                  int device_resident, int64_t chunk_elems, void *stream,
                  double *norm_out);

/* Norm, clip coefficient and non-finite flag of the last finished norm pass
 * on this context (waits for the context's pending work). */
SDP_API int sdp_ctx_last_norm(sdp_ctx *ctx, double *norm, double *clip_coef, int *nonfinite);

/* The BF16 re-emit on its own: dst[i] = bf16_rne(src[i]) for n elements of
 * device memory (the same device routine the fused update uses).  NaN keeps
 * its sign and top payload bits and gets the quiet bit. */
SDP_API int sdp_cast_bf16(sdp_ctx *ctx, const float *src, uint16_t *dst, int64_t n, void *stream);

/* ---- parameter delivery ------------------------------------------------ */

/* How sdp_deliver_params makes the BF16 copy. */
#define SDP_DELIVER_HOST_CAST 0   /* host threads round to BF16 into pinned bounce buffers; BF16 crosses the link */
#define SDP_DELIVER_DEVICE_CAST 1 /* the FP32 chunk crosses the link and the GPU rounds it */

/* Parameter delivery for the next forward pass: dev_bf16[i] = bf16_rne(
 * host_master[i]) for n elements, chunk by chunk, double-buffered.  The paper
 * keeps only the FP32 master on the host and casts each chunk to BF16 while
 * the DMA moves the previous one (Design, overlap within a layer); that is
 * SDP_DELIVER_HOST_CAST.  host_master: any host memory (pinned memory is
 * copied directly in SDP_DELIVER_DEVICE_CAST); dev_bf16: device memory of
 * ctx's GPU.  chunk_elems as for sdp_stream_step.  Blocks until the last
 * chunk has landed, so a forward pass started after the call sees the
 * updated weights (the per-layer version gate).  The first call creates
 * the context's host threads and its two pinned stage buffers (4 *
 * max_chunk_elems bytes each, shared with sdp_host_update_step) if it has
 * none. */
SDP_API int sdp_deliver_params(sdp_ctx *ctx, const float *host_master, uint16_t *dev_bf16, int64_t n,
                       int64_t chunk_elems, int mode);

/* Parameter delivery with the version gate on the GPU instead of the host:
 * as sdp_deliver_params, but the call returns once every chunk is enqueued
 * (in SDP_DELIVER_HOST_CAST mode, once the host threads have rounded the
 * last chunk), and work enqueued on `consumer_stream` (a hipStream_t of
 * ctx's GPU; NULL is the null stream) after this call waits until the last
 * copy has landed.  This is the paper's gate, where dispatch of layer l at
 * iteration t+1 waits for that layer's update from iteration t (Design,
 * completion and buffer reuse).  The caller must keep dev_bf16 alive until
 * then.  In
 * SDP_DELIVER_DEVICE_CAST mode with pinned host_master the DMA reads
 * host_master after the call returns: leave it unchanged until the gate
 * has passed.  Later calls on the context are ordered after this one. */
SDP_API int sdp_deliver_params_async(sdp_ctx *ctx, const float *host_master, uint16_t *dev_bf16,
                                     int64_t n, int64_t chunk_elems, int mode,
                                     void *consumer_stream);

/* The BF16 rounding of the host delivery lane on its own: dst[i] =
 * bf16_rne(src[i]) for n elements of host memory.  ctx may be NULL (runs on
 * the calling thread, no GPU needed) or a context whose host threads share
 * the work. */
SDP_API int sdp_cast_bf16_host(sdp_ctx *ctx, const float *src, uint16_t *dst, int64_t n);

/* ---- step-time model (host only, no GPU needed) --------------------------- */

/* Measured rates that the model takes (each from the library's probes or
 * kernel timing on the machine to be predicted). */
typedef struct {
    double h2d_gbs, d2h_gbs; /* pinned host link, each direction alone (GB/s) */
    double both_gbs;         /* the same, both directions at once (sum of the two) */
    double copy_cmd_us;      /* fixed cost of one copy command */
    double norm_gbs;         /* norm pass and mean-gradient kernel, HBM GB/s */
    double update_gbs;       /* fused update kernel, HBM GB/s */
    double launch_us;        /* fixed cost of one kernel */
    double sync_us;          /* host round trip of the norm read-back; also the delay before a
                                host thread waiting on a GPU command learns that it ended */
    double host_gbs;         /* host memory bandwidth of the host threads' copies (read + written) */
    double host_task_us;     /* fixed cost of one hand-off to the host threads */
    double host_adam_gbs;    /* the host AdamW lane alone (bytes read + written) */
    double dep_us;           /* latency of an event recorded on the copy stream and waited on
                                by the compute stream, or the other way round */
    double dma_host_cost;    /* host memory bandwidth a host task loses per byte of DMA in
                                flight (1: the DMA's own bytes; measured from the host AdamW
                                lane beside a device-to-host copy) */
    double host_issue_us;    /* host-update route: the calling thread's time to enqueue one
                                piece's mean-gradient kernel and copy */
} sdp_rates;

/* What the model predicts for one call. */
typedef struct {
    double predicted_ms; /* finish time of the modelled schedule */
    double bound_ms;     /* resource lower bound: the largest of the six below */
    double h2d_ms, d2h_ms; /* link bytes of each direction / its rate alone */
    double link_ms;      /* all link bytes / the bidirectional rate */
    double gpu_ms;       /* sum of the kernels' modelled times */
    double host_ms;      /* sum of the host-thread tasks' times, each alone */
    double dram_ms;      /* host-task bytes plus every DMA byte / host_gbs */
    int64_t n_chunks;
} sdp_prediction;

/* Schedules the model covers. */
#define SDP_SCHED_STREAMED 0        /* sdp_stream_step, pinned host states */
#define SDP_SCHED_STREAMED_STAGED 1 /* sdp_stream_step with SDP_FLAG_STREAM_STAGED */
#define SDP_SCHED_HOST_ROUTE_F32 2  /* sdp_host_update_step, SDP_GBAR_F32 */
#define SDP_SCHED_HOST_ROUTE_BF16 3 /* sdp_host_update_step, SDP_GBAR_BF16 */

/* Step time of one call on segments of the given sizes, R ranks, chunk_elems
 * and context flags (the g_bar policy of streamed mode and
 * SDP_FLAG_STREAM_HOST_CAST matter).  The
 * paper's step-time model (Design, step-time model) pairs a resource lower
 * bound, max_j W_j / beta_j, with a dependency recurrence f(v) = d_v +
 * max(a_v, f(u) over predecessors u), whose edges are data dependences,
 * stream order and buffer release.  The model builds that graph for the
 * library's own issue order -- each copy, kernel and host-thread task on its
 * stream, each event wait as an edge -- and evaluates it; copies share the
 * link by a fluid model (a direction alone moves at its own rate, both
 * directions together at the bidirectional rate, split in proportion), and
 * host-thread tasks share host memory with the DMA (a task moves at most
 * host_gbs minus dma_host_cost times the copies' current rate, and at most
 * its own rate); a host thread waiting on a GPU command starts sync_us after
 * the command ends. */
SDP_API int sdp_predict_step(int schedule, const int64_t *numels, int32_t n_segs, int32_t n_ranks,
                     int64_t chunk_elems, uint32_t flags, const sdp_rates *rates,
                     sdp_prediction *out);

/* Chunk tuning (the paper's AutoPolicy tunes chunk sizes; Design, automatic
 * policy): the candidate (each a positive multiple of SDP_NORM_TILE) with the
 * smallest predicted step time, the first one on a tie; predicted_ms_out, if
 * not NULL, receives every candidate's prediction. */
SDP_API int sdp_tune_chunk(int schedule, const int64_t *numels, int32_t n_segs, int32_t n_ranks,
                   uint32_t flags, const sdp_rates *rates, const int64_t *candidates,
                   int32_t n_candidates, int64_t *best_out, double *predicted_ms_out);

/* ---- planning (host only, no GPU needed) --------------------------------- */

/* Chunks and norm tiles of a call: n_chunks = sum over segments of
 * ceil(numel / chunk_elems), n_tiles = sum of ceil(numel / SDP_NORM_TILE). */
SDP_API int sdp_plan(const int64_t *numels, int32_t n_segs, int64_t chunk_elems,
             int64_t *n_chunks_out, int64_t *n_tiles_out);

/* Algorithmic bytes per element of one step: device mode HBM traffic, or
 * streamed mode host-link traffic per direction (h2d, d2h), for R ranks and
 * the given context flags' g_bar policy (and, streamed, whether the BF16
 * parameters are rounded on the host: SDP_FLAG_STREAM_HOST_CAST). */
SDP_API int sdp_bytes_per_elem(int streamed, int32_t n_ranks, uint32_t flags,
                       double *hbm_or_h2d, double *d2h);

/* ---- measurement support ---------------------------------------------- */

/* Start (enable = 1, also clears) or stop (0) per-kernel event timing.
 * Starting also creates 256 events in advance, so that timed calls do not
 * spend host time creating them (more are created when needed). */
SDP_API int sdp_ctx_set_timing(sdp_ctx *ctx, int enable);
/* Sum of the recorded kernel times (waits for the recorded events). */
SDP_API int sdp_ctx_get_timing(sdp_ctx *ctx, sdp_kernel_times *out);

/* Device-to-device copy of `bytes` (a multiple of 16) with the library's
 * 16-byte-per-lane streaming pattern: the HBM ceiling and the scale for
 * hardware traffic counters. */
SDP_API int sdp_probe_copy(sdp_ctx *ctx, void *dst, const void *src, int64_t bytes, void *stream);

/* The runtime's own device-to-device copy (hipMemcpyAsync) of `bytes`
 * bytes on `stream`: a second, independent HBM copy ceiling beside
 * sdp_probe_copy.  Device memory of ctx's GPU, not overlapping. */
SDP_API int sdp_probe_memcpy(sdp_ctx *ctx, void *dst, const void *src, int64_t bytes, void *stream);

/* The fused update's memory access pattern with trivial arithmetic, on one
 * device-mode segment (validated as for sdp_agg_adam_step): the same loads
 * and stores, widths and lane mapping, FP32 adds instead of AdamW; from the
 * R gradients, or from stored g_bar (the context's workspace) where the
 * context's device mode stores it (R > 4 by default).  Its rate is the HBM
 * ceiling of the update's own traffic mix.  Measurement only: it overwrites
 * the segment's states and BF16 params.  Asynchronous on `stream`. */
SDP_API int sdp_probe_update_pattern(sdp_ctx *ctx, const sdp_segment *seg, void *stream);

/* The norm pass's memory access pattern when it stores the mean gradient,
 * with trivial arithmetic, on one device-mode segment's gradients (validated
 * as for sdp_agg_adam_step; the states are not touched): the same grid, lane
 * mapping, loads, 16-byte stores and span pairs, into the context's own
 * workspace, under the same residency cap.  Its rate is the HBM ceiling of
 * that pass's traffic mix (2R bytes read and 4 written per element).
 * Measurement only; ordered after the context's previous call, asynchronous
 * on `stream`. */
SDP_API int sdp_probe_norm_pattern(sdp_ctx *ctx, const sdp_segment *seg, void *stream);

/* Pinned host link bandwidth with the streamed engine's copy path:
 * hipMemcpyAsync in chunk_bytes pieces over `bytes`, `reps` times, host to
 * device on the context's copy stream and device to host on its compute
 * stream; when both run, their chunks are issued interleaved, as the engine
 * issues them.  Each figure is timed on the host from the first enqueue to
 * the end of both streams.  gbs_out[0] = H2D alone, [1] = D2H alone,
 * [2] = H2D and D2H at once (sum of both directions).  host_a/host_b:
 * pinned host buffers, dev_a/dev_b: device buffers, each of at least
 * `bytes`.  Blocks. */
SDP_API int sdp_probe_link(sdp_ctx *ctx, void *host_a, void *host_b, void *dev_a, void *dev_b,
                   int64_t bytes, int64_t chunk_bytes, int32_t reps, double *gbs_out);

/* The same link probe on the streamed engine's other device-to-host path:
 * as sdp_probe_link, but each device-to-host piece of chunk_bytes is one
 * launch of the library's copy kernel on the compute stream, storing
 * straight into host_b through its device mapping, as the engine moves a
 * chunk's copies of up to 64 MiB (32 blocks per launch, or
 * SDP_D2H_KERNEL_BLOCKS as read at context creation).  Host-to-device
 * pieces are runtime copies as in sdp_probe_link.  gbs_out[0] = H2D alone,
 * [1] = D2H alone (copy kernel), [2] = both at once (sum).  host_b must be
 * hipHostMalloc memory; dev_b, host_b and chunk_bytes 16-byte aligned.  The
 * streamed mode's link bound takes, per direction and for both at once, the
 * faster of the two probes (the paper's resource lower bound needs the rate
 * of the path the engine can use; Design, step-time model).  Blocks. */
SDP_API int sdp_probe_link_kernel(sdp_ctx *ctx, void *host_a, void *host_b, void *dev_a, void *dev_b,
                                  int64_t bytes, int64_t chunk_bytes, int32_t reps, double *gbs_out);

/* Host memory bandwidth of the context's host threads: `bytes` copied from
 * src to dst (host memory, disjoint) `reps` times in 4 MiB pieces over the
 * threads; gbs_out = bytes read plus bytes written per second / 1e9.  The
 * ceiling of the host lanes (bounce copies, host cast, host AdamW).  Blocks;
 * no GPU work. */
SDP_API int sdp_probe_host_copy(sdp_ctx *ctx, void *dst, const void *src, int64_t bytes, int32_t reps,
                        double *gbs_out);

/* Pinned host memory of exactly `bytes` (hipHostMalloc), for streamed-mode
 * states; free with sdp_host_free. */
SDP_API int sdp_host_alloc(void **out, size_t bytes);
SDP_API int sdp_host_free(void *p);

/* ---- errors ------------------------------------------------------------ */
SDP_API const char *sdp_status_string(int status);
SDP_API const char *sdp_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SDP_H */
