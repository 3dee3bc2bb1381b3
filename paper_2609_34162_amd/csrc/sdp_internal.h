// Internal interface between the C ABI (sdp_runtime.hip) and the gfx950
// kernels (sdp_kernels.hip).  Not installed; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sdp.h"

namespace sdp {

// Result of the norm pass, kept in device memory so that the update kernel
// reads the clip coefficient without a host round trip.
struct NormState {
    double sumsq;
    double norm;
    double clip;
    int32_t nonfinite;
    int32_t pad;
};

// One launch of the norm pass: `n` elements starting at a tile boundary of
// a segment.  The grid is kNormSplit blocks per tile; block b covers the
// elements [b*kNormSpan, min((b+1)*kNormSpan, n)) (none, past the end) and
// writes the double-double pair partials[2b], partials[2b+1], so the tile k
// of the launch owns pairs kNormSplit*k .. kNormSplit*k + kNormSplit - 1.
// When gbar_out is non-null it also stores g_bar there.
struct NormArgs {
    const uint16_t *g[SDP_MAX_RANKS];
    int64_t n;
    double *partials;
    float *gbar_out;
};

// One launch of the fused update over `n` elements.  Gradients come either
// from the R BF16 buffers or, when gbar is non-null, from stored g_bar.
struct UpdateArgs {
    float *p, *m, *v;
    uint16_t *pb;
    const uint16_t *g[SDP_MAX_RANKS];
    const float *gbar;
    int64_t n;
    const NormState *ns;
    // per-step constants, computed once on the host in FP64
    double lr_wd;      // lr * weight_decay
    double beta1, one_minus_beta1;
    double beta2, one_minus_beta2;
    double step_size;  // lr / (1 - beta1^t)
    double inv_bc2;    // 1 / (1 - beta2^t)
    double eps;
};

// One launch of the mean-gradient kernel of the host-update route: g_bar of
// `n` elements from the R BF16 buffers, written to `out` as FP32 or, when
// bf16 is set, rounded to BF16.
struct GbarArgs {
    const uint16_t *g[SDP_MAX_RANKS];
    int64_t n;
    void *out;
    int bf16;
};

// Up to kCopyBatchMax copies of `bytes[k]` bytes from src[k] to dst[k] in
// one launch (the streamed engine's device-to-host copies of a chunk; dst
// may be pinned host memory).  Every dst and src is 16-byte aligned; any
// byte count.
constexpr int kCopyBatchMax = 8;
struct CopyBatch {
    int32_t n;
    char *dst[kCopyBatchMax];
    const char *src[kCopyBatchMax];
    int64_t bytes[kCopyBatchMax];
};

constexpr int kTile = SDP_NORM_TILE;
constexpr int kNormSplit = 16;                   // norm blocks, and partial pairs, per tile
constexpr int kNormSpan = kTile / kNormSplit;    // elements per norm block
constexpr int kNormThreads = 256;
constexpr int kFinalizeThreads = 1024;
// More than kMergeRun span pairs are merged in two fixed stages: block b of
// k_norm_merge merges pairs b*kMergeRun .. (b+1)*kMergeRun - 1 into pair b
// of a second array, and the one-block finalize merges those.
constexpr int kMergeThreads = 256;
constexpr int kMergeRun = 2048;
constexpr int kUpdateThreads = 64;
// Fused update residency: blocks of one wave, at most kUpdateBlocksPerCU of
// them per compute unit (two or three waves per SIMD).  The update's mix of
// seven read and four write streams runs faster with fewer waves in flight
// than the registers would allow; the cap is imposed with dynamic LDS that
// the kernel does not use (the LDS of a compute unit divided by the cap, per
// block).
constexpr int kUpdateBlocksPerCU = 10;
// The norm pass that stores g_bar (16 B read + 4 B written per element at
// R = 8) is capped the same way at kNormStoreBlocksPerCU blocks of
// kNormThreads; the plain norm pass, read only, runs uncapped.
constexpr int kNormStoreBlocksPerCU = 4;
constexpr int kVec = 8;     // elements per lane per access (16 B of BF16, 32 B of FP32)
constexpr int kUpdVec = 4;  // fused update: elements per lane (8 B of BF16, 16 B of FP32)

hipError_t launch_norm_partials(int R, const NormArgs &a, int store_lds_pad, hipStream_t s);
// merged: room for ceil(n_pairs / kMergeRun) pairs (used when n_pairs > kMergeRun).
hipError_t launch_norm_finalize(const double *partials /* pairs */, int64_t n_pairs, double *merged,
                                double max_grad_norm, NormState *ns, hipStream_t s);
hipError_t launch_update(int R, const UpdateArgs &a, int max_blocks, int lds_pad, hipStream_t s);
hipError_t launch_gbar_out(int R, const GbarArgs &a, hipStream_t s);
hipError_t launch_update_pattern(int R, const UpdateArgs &a, int lds_pad, hipStream_t s);
hipError_t launch_norm_pattern(int R, const NormArgs &a, int store_lds_pad, hipStream_t s);
hipError_t launch_cast_bf16(const float *src, uint16_t *dst, int64_t n, hipStream_t s);
hipError_t launch_copy16(void *dst, const void *src, int64_t n16, int max_blocks, hipStream_t s);
// blocks_per_copy: blocks given to each copy of the batch (at most; fewer
// when a copy is short).
hipError_t launch_copy_batch(const CopyBatch &b, int blocks_per_copy, hipStream_t s);
hipError_t launch_fill_u32(void *dst, int64_t n_words, uint32_t value, hipStream_t s);
// One wave that sleeps `sleeps` times for about 64 x 64 clocks each (a fixed
// count: it always ends); the debug jitter's delay on a stream.
hipError_t launch_sleep(int sleeps, hipStream_t s);

}  // namespace sdp
