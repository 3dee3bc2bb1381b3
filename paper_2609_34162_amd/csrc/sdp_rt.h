// Internals shared by the runtime's translation units: sdp_runtime.hip (the
// context, validation, device mode, measurement and the step-time model's C
// entry points), sdp_stream.hip (the streamed engine) and
// sdp_host_route.hip (parameter delivery and the host-update route).  Not
// installed; not part of the ABI.
#pragma once

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <limits>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include <pthread.h>
#include <sched.h>

#include "sdp_host.h"
#include "sdp_internal.h"

namespace sdprt {

using sdp::NormState;

// Detail of the last failure on the calling thread (sdp_last_error()).
extern thread_local std::string t_err;

// Records the detail and returns `status`.
int fail(int status, const char *fmt, ...);

#define HIP_TRY(expr)                                                                        \
    do {                                                                                     \
        hipError_t e_ = (expr);                                                              \
        if (e_ != hipSuccess)                                                                \
            return fail(SDP_ERR_HIP, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(e_),   \
                        __FILE__, __LINE__);                                                 \
    } while (0)

#define SDP_TRY(expr)              \
    do {                           \
        int rc_ = (expr);          \
        if (rc_ != SDP_OK) return rc_; \
    } while (0)

// ceil(a / b) for a >= 0, b > 0, without overflow near the int64 limit
inline int64_t cdiv(int64_t a, int64_t b) { return a / b + (a % b != 0); }
inline int64_t round_up(int64_t a, int64_t b) { return cdiv(a, b) * b; }

struct DeviceGuard {
    int old = -1;
    explicit DeviceGuard(int d) {
        if (hipGetDevice(&old) != hipSuccess) old = -1;
        if (old != d) (void)hipSetDevice(d);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (old >= 0 && hipGetDevice(&cur) == hipSuccess && cur != old) (void)hipSetDevice(old);
    }
};

enum TimedKind { kNorm = 0, kFinalize = 1, kUpdate = 2, kGbar = 3 };

struct Timed {
    int kind;
    hipEvent_t a, b;
    int64_t elems;
};

// Round FP32 values to BF16, nearest even, on the host (the parameter
// delivery lane).  NaN keeps its sign and top payload bits and gets the quiet
// bit; infinities are kept; overflow of the largest values rounds to
// infinity.  Plain integer code that the compiler vectorises.
void cast_bf16_host(const float *src, uint16_t *dst, size_t n);

// A fixed set of host threads for the host lanes: copies between the
// caller's memory and the staged mode's pinned bounce buffers (the CPU-side
// staging lane of the paper's chunked overlap, Design, overlap within a
// layer), the BF16 rounding of parameter delivery and the host AdamW of the
// host-update route.  run(n, fn) calls fn(i) for every i in [0, n) across
// the workers and the caller.
class HostPool {
  public:
    // pin: worker i stays on the (i+1)-th CPU of the process's affinity set
    // (cyclically), leaving the first to the calling thread.
    HostPool(int workers, bool pin) {
        std::vector<int> cpus;
        if (pin) {
            cpu_set_t set;
            CPU_ZERO(&set);
            if (sched_getaffinity(0, sizeof set, &set) == 0)
                for (int c = 0; c < CPU_SETSIZE; ++c)
                    if (CPU_ISSET(c, &set)) cpus.push_back(c);
        }
        for (int i = 0; i < workers; ++i) {
            const int cpu = cpus.empty() ? -1 : cpus[(size_t)(i + 1) % cpus.size()];
            threads_.emplace_back([this, cpu, i] {
                if (cpu >= 0) {
                    cpu_set_t one;
                    CPU_ZERO(&one);
                    CPU_SET(cpu, &one);
                    (void)pthread_setaffinity_np(pthread_self(), sizeof one, &one);
                }
                loop(i);
            });
        }
    }
    ~HostPool() {
        {
            std::lock_guard<std::mutex> g(mu_);
            stop_ = true;
        }
        cv_work_.notify_all();
        for (auto &t : threads_) t.join();
    }
    int size() const { return (int)threads_.size() + 1; }

    // Runs fn(0) .. fn(n-1) on the calling thread and the workers; width > 0
    // limits them to the calling thread and the first width - 1 workers.
    void run(size_t n, const std::function<void(size_t)> &fn, int width = 0) {
        std::unique_lock<std::mutex> g(mu_);
        fn_ = &fn;
        n_ = n;
        next_ = 0;
        left_ = n;
        width_ = width > 0 ? width : size();
        ++gen_;
        g.unlock();
        cv_work_.notify_all();
        work();
        g.lock();
        cv_done_.wait(g, [this] { return left_ == 0; });
        fn_ = nullptr;
    }

  private:
    void work() {
        for (;;) {
            size_t k;
            const std::function<void(size_t)> *fn;
            {
                std::lock_guard<std::mutex> g(mu_);
                if (next_ >= n_) return;
                k = next_++;
                fn = fn_;
            }
            (*fn)(k);
            std::lock_guard<std::mutex> g(mu_);
            if (--left_ == 0) cv_done_.notify_all();
        }
    }
    void loop(int index) {
        uint64_t seen = 0;
        for (;;) {
            bool join;
            {
                std::unique_lock<std::mutex> g(mu_);
                cv_work_.wait(g, [&] { return stop_ || gen_ != seen; });
                if (stop_) return;
                seen = gen_;
                join = index + 1 < width_;
            }
            if (join) work();
        }
    }

    std::vector<std::thread> threads_;
    std::mutex mu_;
    std::condition_variable cv_work_, cv_done_;
    const std::function<void(size_t)> *fn_ = nullptr;
    size_t n_ = 0, next_ = 0, left_ = 0;
    int width_ = 0;
    uint64_t gen_ = 0;
    bool stop_ = false;
};

// Copies (kind kCopy: `bytes`) and BF16 roundings (kind kCastBf16: `bytes`
// FP32 values at src into BF16 at dst), split into pieces over the pool.
struct Job {
    enum Kind { kCopy = 0, kCastBf16 = 1 };
    void *dst;
    const void *src;
    size_t bytes;
    int kind = kCopy;
};

// width > 0: on at most that many threads (see HostPool::run).
void pool_jobs(HostPool *pool, const std::vector<Job> &jobs, int width = 0);

// Staged mode: bounce buffers.  Incoming chunks rotate over kInBufs pinned
// buffers shaped like a slot, outgoing results over kOutBufs buffers of
// 14 * max_chunk bytes.  In the update phase the host thread stages and
// enqueues chunk j + kStageAhead before it drains chunk j, and drains each
// chunk as soon as its results have landed.  Staging only one chunk ahead
// put the host copies of a chunk (its drain, then the next chunk's staging)
// between two device-to-host copies, so each chunk waited for them.  Chunk
// j + kStageAhead lands in outgoing buffer (j + kStageAhead) % kOutBufs,
// which chunk j + kStageAhead - kOutBufs used and the host has drained.
constexpr int kInBufs = 3;
constexpr int kOutBufs = 3;
constexpr int kStageAhead = 2;
static_assert(kStageAhead < kInBufs && kStageAhead < kOutBufs, "staging ahead needs free bounce buffers");

// A host <-> staging-slot transfer of one chunk: `bytes` at byte offset `off`
// of a slot, from or to `host`.
struct Xfer {
    size_t off;
    char *host;
    size_t bytes;
};

}  // namespace sdprt

// The context behind the opaque sdp_ctx of the ABI.
struct sdp_ctx {
    int device = 0;
    int64_t max_chunk = 0;
    int32_t max_ranks = 0;
    uint32_t flags = 0;
    uint64_t jitter_state = 0;  // SDP_FLAG_DEBUG_JITTER's generator (xorshift64*)
    hipStream_t s_copy = nullptr, s_comp = nullptr;
    hipEvent_t h2d_done[2] = {nullptr, nullptr};
    hipEvent_t slot_free[2] = {nullptr, nullptr};
    hipEvent_t last_done = nullptr;
    hipEvent_t copy_done = nullptr;  // copy stream's last work of a gated delivery
    bool last_done_valid = false;
    char *staging = nullptr;
    size_t slot_bytes = 0;
    // staged streamed mode: pinned bounce buffers shaped like the slots
    char *bounce_in = nullptr;   // kInBufs x slot_bytes
    char *bounce_out = nullptr;  // kOutBufs x 14 * max_chunk (master, m, v, bf16 part of a slot)
    ptrdiff_t bounce_out_map = 0;  // device mapping of bounce_out minus its host address
    hipEvent_t bin_done[sdprt::kInBufs] = {};   // copy stream: the copies out of bounce_in[k] are done
    hipEvent_t d2h_done[sdprt::kOutBufs] = {};  // compute stream: the copies into bounce_out[k] are done
    bool bin_used[sdprt::kInBufs] = {};
    // parameter delivery and the host-update route: two pinned buffers of
    // 4 * max_chunk bytes each (one chunk of FP32), created on first use
    char *stage = nullptr;
    ptrdiff_t stage_map = 0;  // device mapping of stage minus its host address
    bool stage_used[2] = {false, false};
    std::vector<sdprt::Xfer> pending_out[sdprt::kOutBufs];
    // SDP_FLAG_STREAM_HOST_CAST: the BF16 rounding of each chunk whose master
    // lands with outgoing copies `bo`, run once they have landed
    std::vector<sdprt::Job> pending_cast[sdprt::kOutBufs];
    sdprt::HostPool *copier = nullptr;
    int staged_copy_threads = 0;   // staged update pass: host copy threads while the DMA runs
    int64_t d2h_kernel_max = 0;    // device-to-host copies up to this many bytes run as k_copy_batch
    int d2h_kernel_blocks = 0;     // blocks per copy of such a launch (0: kD2HLaunchBlocks spread over the copies)
    double *partials = nullptr;
    int64_t partials_cap = 0;
    float *gbar = nullptr;
    int64_t gbar_cap = 0;
    sdp::NormState *ns = nullptr;       // device
    sdp::NormState *ns_host = nullptr;  // pinned mirror for read-back
    int update_max_blocks = 0;     // 0: one 8-element group per lane
    int update_lds_pad = 0;        // dynamic LDS bytes per update block (residency cap); 0: no cap
    int norm_store_lds_pad = 0;    // the same for the norm pass that stores g_bar
    bool timing = false;
    std::vector<sdprt::Timed> timed;
    // host lanes of the host-update route, timed on the host clock
    double host_adam_ms = 0.0, host_wait_ms = 0.0, host_issue_ms = 0.0;
    int64_t host_issues = 0;
    int64_t host_adam_elems = 0;
    std::vector<hipEvent_t> pool;
};

namespace sdprt {

// ---- validation ---------------------------------------------------------

int check_hparams(const sdp_adamw_params *hp);
inline bool aligned(const void *p) { return ((uintptr_t)p % SDP_ALIGN) == 0; }
int check_device_ptr(const sdp_ctx *ctx, const void *p, size_t bytes, const char *what, int seg);
int check_pinned_ptr(const void *p, size_t bytes, const char *what, int seg);
int check_host_ptr(const void *p, const char *what, int seg);
enum MemKind { kDeviceMem, kPinnedHost, kAnyHost };
struct Range {
    uintptr_t a, b;
    int seg;
    const char *what;
};
inline bool overlap(const Range &x, const Range &y) { return x.a < y.b && y.a < x.b; }
int validate_segments(const sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, MemKind state_kind,
                      MemKind grad_kind, bool grads_only, int32_t *R_out);
int check_chunk(int64_t chunk, bool allow_zero);

// ---- workspace ----------------------------------------------------------

int ensure_partials(sdp_ctx *ctx, int64_t tiles);
double *tile_partials(sdp_ctx *ctx, int64_t tile);  // the first pair of a tile's span partials
int ensure_gbar(sdp_ctx *ctx, int64_t n);
// Layout of one call: norm tiles and stored-g_bar offsets of each segment.
struct Plan {
    std::vector<int64_t> tile_base, gbar_base;
    int64_t tiles = 0, gbar_elems = 0;
};
Plan make_plan(const sdp_segment *segs, int32_t n_segs);
bool device_gbar(const sdp_ctx *ctx, int32_t R);

// ---- timing -------------------------------------------------------------

hipEvent_t take_event(sdp_ctx *ctx);
hipEvent_t timed_begin(sdp_ctx *ctx, hipStream_t s);
void timed_end(sdp_ctx *ctx, hipStream_t s, hipEvent_t a, int kind, int64_t elems);

// ---- launches and ordering shared by the modes ---------------------------

int norm_launch(sdp_ctx *ctx, int32_t R, const uint16_t *const *g, int64_t n, double *partials, float *gbar_out,
                hipStream_t s);
int finalize_launch(sdp_ctx *ctx, int64_t tiles, double max_grad_norm, hipStream_t s);
void fill_consts(const sdp_adamw_params *hp, sdp::UpdateArgs &a);
int update_launch(sdp_ctx *ctx, int32_t R, const sdp_adamw_params *hp, float *p, float *m, float *v, uint16_t *pb,
                  const uint16_t *const *g, const float *gbar, int64_t n, hipStream_t s);
int order_after_last(sdp_ctx *ctx, hipStream_t s);
int mark_done(sdp_ctx *ctx, hipStream_t s);
int read_norm(sdp_ctx *ctx, hipStream_t s, NormState *out);
int device_norm(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int32_t R, const Plan &plan, bool store_gbar,
                double max_grad_norm, hipStream_t s);
int sync_streams(sdp_ctx *ctx);

// SDP_FLAG_DEBUG_JITTER: a random delay of 0-200 us enqueued on stream s
// (jitter_stream), or slept by the calling thread (jitter_host); nothing
// without the flag.
int jitter_stream(sdp_ctx *ctx, hipStream_t s);
void jitter_host(sdp_ctx *ctx);

// ---- chunks and staging slots -------------------------------------------

struct Slot {
    float *p, *m, *v;
    uint16_t *pb;
    uint16_t *g[SDP_MAX_RANKS];
};
Slot slot_at(const sdp_ctx *ctx, int k);
struct Chunk {
    int32_t seg;
    int64_t off, len;
};
std::vector<Chunk> make_chunks(const sdp_segment *segs, int32_t n_segs, int64_t C);
inline bool staged(const sdp_ctx *ctx) { return (ctx->flags & SDP_FLAG_STREAM_STAGED) != 0; }
inline bool host_cast(const sdp_ctx *ctx) { return (ctx->flags & SDP_FLAG_STREAM_HOST_CAST) != 0; }
size_t off_in_slot(const sdp_ctx *ctx, int sl, const void *p);
int stream_common_checks(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int64_t chunk, bool grads_only,
                         int32_t *R);
int stream_norm_phase(sdp_ctx *ctx, const sdp_segment *segs, int32_t n_segs, int32_t R, const Plan &plan,
                      const std::vector<Chunk> &chunks, bool store_gbar, double max_grad_norm, bool used[2]);

// ---- host threads and pinned stage buffers ------------------------------

int default_host_threads();
// Staged update pass: how many host threads copy into and out of the bounce
// buffers while copies in both directions are in flight.  Host memory
// carries those copies and every DMA byte; on the MI355X hosts measured here
// (about 400 GB/s of host memory traffic with 16 threads, 50-57 GB/s per
// thread) four and five threads let the DMA keep its rate, and six or more
// starved the device-to-host copies and slowed the pass by a quarter; the
// default keeps one thread of margin below that cliff.
constexpr int kStagedCopyThreads = 4;
int default_staged_copy_threads();

// Streamed engine: device-to-host copies of at most kD2HKernelMaxBytes run as
// the library's own copy kernel.  The runtime moves copies of a few MiB with
// DMA copy commands that measured 10-45 GB/s beside host-to-device traffic;
// larger ones it moves with copy kernels that reach the link's rate.  A
// launch spreads kD2HLaunchBlocks blocks over its copies, at least
// kD2HMinBlocksPerCopy each: on the Qwen3-14B layer about 32 blocks writing
// to host memory at once were fastest (8 per copy for four copies, 32 for
// one), and 64 per copy cost up to 1% of the step.
constexpr int64_t kD2HKernelMaxBytes = 64ll << 20;
constexpr int kD2HLaunchBlocks = 32;
constexpr int kD2HMinBlocksPerCopy = 8;
// Device -> pinned host copies (dst <- src, bytes) enqueued on stream st,
// through the copy kernel where they qualify (sdp_stream.hip).  own_map:
// NULL, or the offset of the device mapping of the destinations, which are a
// buffer of the context's own (no attribute query then).
int d2h_copies(sdp_ctx *ctx, const std::vector<std::pair<char *, const char *>> &ends,
               const std::vector<size_t> &bytes, hipStream_t st, const ptrdiff_t *own_map);
// Offset of the device's mapping of pinned host memory p from p itself.
int device_map_offset(const void *p, ptrdiff_t *out);
HostPool *new_pool(const sdp_ctx *ctx, int threads);
inline size_t stage_bytes(const sdp_ctx *ctx) { return 4 * (size_t)ctx->max_chunk; }
int ensure_host_stage(sdp_ctx *ctx);
bool is_pinned_host(const void *p);
using Clock = std::chrono::steady_clock;
inline double ms_between(Clock::time_point a, Clock::time_point b) {
    return std::chrono::duration<double, std::milli>(b - a).count();
}

}  // namespace sdprt
