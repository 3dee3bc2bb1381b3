// gfx950 copy kernel of the streamed engine: a batch of device-to-host
// copies of one chunk (master, exp_avg, exp_avg_sq and BF16 parameters) in
// one launch, written straight into pinned host memory.  Also the debug
// jitter's sleeping kernel.
#include "sdp_internal.h"

namespace sdp {
namespace {

// Copy k of the batch is blockIdx.y; its blocks stride over its 16-byte
// words, and the first block copies the ragged tail byte by byte.
__global__ __launch_bounds__(256) void k_copy_batch(CopyBatch b) {
    const int k = blockIdx.y;
    const int64_t bytes = b.bytes[k];
    const int64_t n16 = bytes / 16;
    const uint4 *__restrict__ src = reinterpret_cast<const uint4 *>(b.src[k]);
    uint4 *__restrict__ dst = reinterpret_cast<uint4 *>(b.dst[k]);
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride) dst[i] = src[i];
    const int64_t tail = bytes - n16 * 16;
    if (blockIdx.x == 0 && threadIdx.x < tail) b.dst[k][n16 * 16 + threadIdx.x] = b.src[k][n16 * 16 + threadIdx.x];
}

// The debug jitter's delay: a fixed number of s_sleep 64 (about 4,096
// clocks each), then the wave ends.
__global__ __launch_bounds__(64) void k_sleep(int sleeps) {
    for (int i = 0; i < sleeps; ++i) __builtin_amdgcn_s_sleep(64);
}

}  // namespace

hipError_t launch_sleep(int sleeps, hipStream_t s) {
    if (sleeps < 0 || sleeps > 4096) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_sleep, dim3(1), dim3(64), 0, s, sleeps);
    return hipGetLastError();
}

hipError_t launch_copy_batch(const CopyBatch &b, int blocks_per_copy, hipStream_t s) {
    if (b.n < 1 || b.n > kCopyBatchMax || blocks_per_copy < 1) return hipErrorInvalidValue;
    int64_t longest = 0;
    for (int k = 0; k < b.n; ++k) {
        if (b.bytes[k] < 0 || ((uintptr_t)b.dst[k] | (uintptr_t)b.src[k]) % 16 != 0) return hipErrorInvalidValue;
        longest = b.bytes[k] > longest ? b.bytes[k] : longest;
    }
    int64_t blocks = (longest / 16 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > blocks_per_copy) blocks = blocks_per_copy;
    hipLaunchKernelGGL(k_copy_batch, dim3((uint32_t)blocks, (uint32_t)b.n), dim3(256), 0, s, b);
    return hipGetLastError();
}

}  // namespace sdp
