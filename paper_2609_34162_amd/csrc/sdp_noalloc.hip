// C ABI of libsdp: device mode for callers that cannot allocate
// (sdp_agg_adam_step_noalloc).  The call's workspace -- the norm pass's span
// partials, the finalize's merge stage and the norm state the fused update
// reads -- lives in one file-scope device array, `scratch`, instead of a
// context's allocations.  Every GPU the library runs on holds its own copy of
// the array until the process ends; its address on each device is looked up
// once (hipGetSymbolAddress, with that device current) and only that address
// is ever handed to a kernel or a copy.  The mean gradient is not stored:
// the update reads the rank gradients again (26 + 4R bytes per element).
//
// Nothing here allocates: no hipMalloc or hipFree, and no host heap (fixed
// arrays on the stack for validation).  Calls on one GPU share its array, so
// calls that overlap on one GPU (different streams, or different host
// threads) race; calls on one stream are ordered.  Each call writes every
// partial, merged pair and the norm state before reading them, so nothing
// needs clearing between calls.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <string>

#include "sdp.h"
#include "sdp_internal.h"

namespace sdprt {
int fail(int status, const char *fmt, ...);
extern thread_local std::string t_err;
int check_hparams(const sdp_adamw_params *hp);
void fill_consts(const sdp_adamw_params *hp, sdp::UpdateArgs &a);
}  // namespace sdprt

namespace {

using sdprt::fail;

#define SDP_TRY_NA(expr)              \
    do {                              \
        const int rc_ = (expr);       \
        if (rc_ != SDP_OK) return rc_; \
    } while (0)

constexpr int64_t kMaxTiles = SDP_NOALLOC_MAX_TILES;
constexpr int64_t kMaxPairs = kMaxTiles * sdp::kNormSplit;
constexpr int64_t kMaxMerged = (kMaxPairs + sdp::kMergeRun - 1) / sdp::kMergeRun;
constexpr size_t kPairBytes = 2 * sizeof(double);
constexpr size_t kNormStateOffset = (size_t)(kMaxPairs + kMaxMerged) * kPairBytes;
constexpr size_t kScratchBytes = kNormStateOffset + 256;
static_assert(sizeof(sdp::NormState) <= 256, "norm state fits its slot");
static_assert(kNormStateOffset % 256 == 0, "norm state 256-byte aligned");

// The workspace of sdp_agg_adam_step_noalloc on each GPU (device memory).
// In host code this name is not a device address: host code uses only the
// address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;

struct DeviceSetup {
    bool ready = false;
    unsigned char *ptr = nullptr;  // scratch on this device
    int update_lds_pad = 0;        // the fused update's residency cap, as a context sets it
};

std::mutex g_setup_mu;
DeviceSetup g_setup[kMaxDevices];

int setup_device(int device, DeviceSetup *out) {
    std::lock_guard<std::mutex> lock(g_setup_mu);
    DeviceSetup &d = g_setup[device];
    if (!d.ready) {
        void *p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(SDP_ERR_HIP, "hipGetSymbolAddress(scratch) on GPU %d failed: %s", device,
                        hipGetErrorString(e));
        }
        int lds_cu = 0, lds_block = 0;
        if (hipDeviceGetAttribute(&lds_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, device) !=
                hipSuccess ||
            hipDeviceGetAttribute(&lds_block, hipDeviceAttributeMaxSharedMemoryPerBlock, device) != hipSuccess) {
            (void)hipGetLastError();
            return fail(SDP_ERR_HIP, "cannot query the LDS size of GPU %d", device);
        }
        // the same cap as a context's default: the compute unit's LDS over
        // kUpdateBlocksPerCU blocks, through dynamic LDS the kernel never uses
        const int pad = (lds_cu / sdp::kUpdateBlocksPerCU) / 1024 * 1024;
        d.update_lds_pad = pad > 0 && pad <= lds_block ? pad : 0;
        d.ptr = (unsigned char *)p;
        d.ready = true;
    }
    *out = d;
    return SDP_OK;
}

struct Span {
    uintptr_t a, b;
    int seg;
    const char *what;
};

// Device memory of `device` covering [p, p + bytes) within one allocation.
int check_dev(int device, const void *p, size_t bytes, const char *what, int seg) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s (%p) is not device memory", seg, what, p);
    }
    if (at.type != hipMemoryTypeDevice || at.device != device)
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s (%p) is not device memory of GPU %d", seg, what, p,
                    device);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p) != hipSuccess) {
        (void)hipGetLastError();
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s (%p): allocation range unknown", seg, what, p);
    }
    if ((const char *)p + bytes > (const char *)base + size)
        return fail(SDP_ERR_NOT_DEVICE_MEMORY, "segment %d %s: %zu bytes at %p overrun its allocation", seg, what,
                    bytes, p);
    return SDP_OK;
}

}  // namespace

extern "C" {

int sdp_agg_adam_step_noalloc(const sdp_segment *segs, int32_t n_segs, const sdp_adamw_params *hp, void *stream,
                              double *grad_norm_out) {
    sdprt::t_err.clear();
    // sizes first: they need no GPU
    if (!segs || n_segs < 1 || n_segs > SDP_NOALLOC_MAX_SEGMENTS)
        return fail(SDP_ERR_INVALID_ARGUMENT, "sdp_agg_adam_step_noalloc: need 1..%d segments (got %d)",
                    SDP_NOALLOC_MAX_SEGMENTS, n_segs);
    int64_t tiles = 0;
    for (int32_t s = 0; s < n_segs; ++s) {
        if (segs[s].numel < 1) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d: numel must be >= 1", s);
        tiles += (segs[s].numel / SDP_NORM_TILE + (segs[s].numel % SDP_NORM_TILE != 0));
        if (tiles > kMaxTiles)
            return fail(SDP_ERR_INVALID_ARGUMENT,
                        "sdp_agg_adam_step_noalloc: the segments need more than %lld norm tiles of %d elements "
                        "(at most %lld elements in all); its static workspace holds %lld",
                        (long long)kMaxTiles, SDP_NORM_TILE, (long long)(kMaxTiles * SDP_NORM_TILE),
                        (long long)kMaxTiles);
    }
    const int32_t R = segs[0].n_ranks;
    if (R < 1 || R > SDP_MAX_RANKS)
        return fail(SDP_ERR_INVALID_ARGUMENT, "n_ranks must be in 1..%d (got %d)", SDP_MAX_RANKS, R);
    SDP_TRY_NA(sdprt::check_hparams(hp));
    int device = 0;
    if (hipGetDevice(&device) != hipSuccess || device < 0 || device >= kMaxDevices) {
        (void)hipGetLastError();
        return fail(SDP_ERR_HIP, "no current GPU (or device index above %d)", kMaxDevices - 1);
    }
    // every buffer: non-NULL, aligned, device memory of this GPU; states
    // pairwise disjoint (sorted on the stack), then, in a second pass, every
    // gradient disjoint from every state
    Span states[4 * SDP_NOALLOC_MAX_SEGMENTS];
    int n_states = 0;
    for (int32_t s = 0; s < n_segs; ++s) {
        const sdp_segment &g = segs[s];
        if (g.n_ranks != R)
            return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d has n_ranks %d, segment 0 has %d", s, g.n_ranks, R);
        if (!g.grads) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d: grads is NULL", s);
        const size_t n = (size_t)g.numel;
        const struct {
            const void *p;
            size_t bytes;
            const char *what;
        } bufs[4] = {{g.master, 4 * n, "master"}, {g.exp_avg, 4 * n, "exp_avg"},
                     {g.exp_avg_sq, 4 * n, "exp_avg_sq"}, {g.param_bf16, 2 * n, "param_bf16"}};
        for (int k = 0; k < 4 + R; ++k) {
            const void *p = k < 4 ? bufs[k].p : (const void *)g.grads[k - 4];
            const size_t bytes = k < 4 ? bufs[k].bytes : 2 * n;
            const char *what = k < 4 ? bufs[k].what : "grad";
            if (!p) return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d: %s is NULL", s, what);
            if ((uintptr_t)p % SDP_ALIGN != 0)
                return fail(SDP_ERR_ALIGNMENT, "segment %d: %s (%p) is not %d-byte aligned", s, what, p, SDP_ALIGN);
            SDP_TRY_NA(check_dev(device, p, bytes, what, s));
            if (k < 4) states[n_states++] = Span{(uintptr_t)p, (uintptr_t)p + bytes, s, what};
        }
    }
    std::sort(states, states + n_states, [](const Span &x, const Span &y) { return x.a < y.a; });
    for (int k = 1; k < n_states; ++k)
        if (states[k - 1].b > states[k].a)
            return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d %s overlaps segment %d %s", states[k - 1].seg,
                        states[k - 1].what, states[k].seg, states[k].what);
    for (int32_t s = 0; s < n_segs; ++s)
        for (int32_t r = 0; r < R; ++r) {
            const uintptr_t a = (uintptr_t)segs[s].grads[r], b = a + 2 * (size_t)segs[s].numel;
            for (int k = 0; k < n_states; ++k)
                if (a < states[k].b && states[k].a < b)
                    return fail(SDP_ERR_INVALID_ARGUMENT, "segment %d gradient overlaps segment %d %s", s,
                                states[k].seg, states[k].what);
        }
    DeviceSetup dev;
    SDP_TRY_NA(setup_device(device, &dev));
    double *partials = reinterpret_cast<double *>(dev.ptr);
    double *merged = partials + 2 * kMaxPairs;
    sdp::NormState *ns = reinterpret_cast<sdp::NormState *>(dev.ptr + kNormStateOffset);
    hipStream_t st = (hipStream_t)stream;
#define NA_HIP(expr)                                                                                   \
    do {                                                                                               \
        hipError_t e_ = (expr);                                                                        \
        if (e_ != hipSuccess) {                                                                        \
            (void)hipGetLastError();                                                                   \
            return fail(SDP_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_));                   \
        }                                                                                              \
    } while (0)
    // norm pass over every tile of every segment, in segment then tile order
    int64_t tile_base = 0;
    for (int32_t s = 0; s < n_segs; ++s) {
        sdp::NormArgs a{};
        for (int32_t r = 0; r < R; ++r) a.g[r] = segs[s].grads[r];
        a.n = segs[s].numel;
        a.partials = partials + 2 * sdp::kNormSplit * tile_base;
        a.gbar_out = nullptr;
        NA_HIP(sdp::launch_norm_partials(R, a, 0, st));
        tile_base += (segs[s].numel / SDP_NORM_TILE + (segs[s].numel % SDP_NORM_TILE != 0));
    }
    NA_HIP(sdp::launch_norm_finalize(partials, tiles * sdp::kNormSplit, merged, hp->max_grad_norm, ns, st));
    // the fused update, reading the clip coefficient from the norm state,
    // with the per-step constants computed as for every other mode
    for (int32_t s = 0; s < n_segs; ++s) {
        const sdp_segment &g = segs[s];
        sdp::UpdateArgs a{};
        a.p = g.master;
        a.m = g.exp_avg;
        a.v = g.exp_avg_sq;
        a.pb = g.param_bf16;
        for (int32_t r = 0; r < R; ++r) a.g[r] = g.grads[r];
        a.gbar = nullptr;
        a.n = g.numel;
        a.ns = ns;
        sdprt::fill_consts(hp, a);
        NA_HIP(sdp::launch_update(R, a, 0, dev.update_lds_pad, st));
    }
    if (grad_norm_out) {
        sdp::NormState hs{};
        NA_HIP(hipMemcpyAsync(&hs, ns, sizeof hs, hipMemcpyDeviceToHost, st));
        NA_HIP(hipStreamSynchronize(st));
        *grad_norm_out = hs.norm;
        if (hs.nonfinite)
            return fail(SDP_ERR_NONFINITE, "gradient norm is not finite (%g); nothing was updated", hs.norm);
    }
#undef NA_HIP
    return SDP_OK;
}

}  // extern "C"
