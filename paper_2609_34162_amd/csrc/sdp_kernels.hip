// gfx950 kernels of the data-parallel update: norm partials over fixed tiles,
// a fixed-order finalize (one block, after a merge stage for many partials),
// and the fused aggregate + clip + AdamW + BF16 re-emit pass.  All of them
// are bound by HBM bandwidth and use no MFMA.
// Their lanes move wide accesses: 16-byte (dwordx4) FP32 accesses throughout,
// and BF16 in 16-byte or 8-byte pieces (eight or four elements per lane).
//
// Element arithmetic (the paper names mixed-precision Adam over FP32 master
// weights and moments, fed by the gradient averaged over the ranks, and BF16
// compute weights; the formulas are AdamW with decoupled decay and
// Kingma-Ba bias correction):
//   g_bar = fp32(S / R), S the exact sum of the R BF16 values, rounded once
//   g     = g_bar * c                               (c from the global norm)
//   p1 = p - lr*wd*p ; m' = b1 m + (1-b1) g ; v' = b2 v + (1-b2) g^2
//   p' = p1 - lr/(1-b1^t) * m' / (sqrt(v'/(1-b2^t)) + eps)
// in FP64 registers, each output rounded once to FP32, BF16 from the FP32.
#include "sdp_internal.h"

namespace sdp {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Streaming accesses: every array of the two passes is touched once per pass
// and is far larger than the 256 MB last-level cache, so the kernels load and
// store with the non-temporal hint (the cache does not keep the lines).
__device__ __forceinline__ float4 load_nt4(const float *p) {
    const f32x4 t = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(p));
    return make_float4(t.x, t.y, t.z, t.w);
}
__device__ __forceinline__ void store_nt4(float *p, float4 v) {
    const f32x4 t = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(t, reinterpret_cast<f32x4 *>(p));
}
__device__ __forceinline__ void store_nt2(uint16_t *p, uint32_t lo, uint32_t hi) {
    const u32x2 t = {lo, hi};
    __builtin_nontemporal_store(t, reinterpret_cast<u32x2 *>(p));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Round to nearest even on the top 16 bits.  NaN: keep sign and top payload
// bits, set the quiet bit (adding the rounding bias could carry a NaN into
// the infinity pattern).  Infinity stays infinity; overflow of the largest
// finite values rounds to infinity as IEEE round-to-nearest does.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x0040u;
    return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    return bf16_rne(lo) | (bf16_rne(hi) << 16);
}

template <int R>
__device__ __forceinline__ float mean_of(double s) {
    // R a power of two: the product by 1/R is exact and equals s / R.
    if constexpr ((R & (R - 1)) == 0) {
        return (float)(s * (1.0 / (double)R));
    } else {
        return (float)(s / (double)R);
    }
}

// ---------------------------------------------------------------------------
// Mean gradient g_bar = fp32(S / R): S, the exact sum of the R BF16 values,
// divided by R and rounded once.
//
// Fast route.  Summed in FP64 (from +0, in rank order), R BF16 values give S
// exactly when their magnitudes are close enough (span_exact below); then
// fp32(fp64(S / R)) is the single rounding of S / R.  Proof: the two
// roundings differ only if fp64(S / R) is an FP32 midpoint m with S / R != m.
// With 2^E <= S / R < 2^(E+1) that needs |S - R m| <= R 2^(E-53).  S - R m is
// a nonzero multiple of the smaller of S's last-bit weight 2^f and 2^(E-24)
// (the grid of R m); 2^(E-24) exceeds R 2^(E-53) for every R < 2^29, so
// 2^f <= R 2^(E-53), and S / 2^f >= R 2^E / (R 2^(E-53)) = 2^53: S would not
// be an FP64 number.  (Below 2^-126 the FP32 grid is 2^-150 and S's last bit
// weighs at least 2^-133, so the same holds.)
//
// Wide route (magnitudes spread over more binades, which the workloads'
// gradients practically never reach): S is summed exactly as a fixed-point
// integer, rounded to odd at 53 bits (truncated, last bit forced to 1 if
// anything was dropped), and that FP64 value takes the fast route's last two
// steps.  Rounding to odd keeps S on the same side of every number of at most
// 52 significant bits; R times an FP32 value or midpoint has at most 30, so
// fp32 of the quotient is unchanged.

// A lane's values sum exactly in FP64, in any order, when the binade of the
// largest magnitude exceeds that of the smallest nonzero one by at most
// 45 - ceil(log2 R): every value is then a multiple of the smallest one's
// last-bit weight u = 2^(max(e_min, 1) - 134), and every partial sum is
// below R 2^(e_max - 126) <= 2^53 u.
template <int R>
constexpr int kExactSpan = 45 - (R <= 1 ? 0 : R <= 2 ? 1 : R <= 4 ? 2 : R <= 8 ? 3 : 4);

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Largest magnitude and smallest nonzero magnitude (minus one) of BF16
// values packed two per word; a zero wraps to 0xffff and so never counts as
// the smallest.
struct Span {
    u16x2 top, low;
};

__device__ __forceinline__ Span span_init() {
    Span s;
    s.top = (u16x2)(0);
    s.low = (u16x2)(0xffff);
    return s;
}

__device__ __forceinline__ void span_add(Span &s, uint32_t word) {
    const u16x2 m = __builtin_bit_cast(u16x2, word & 0x7fff7fffu);
    s.top = __builtin_elementwise_max(s.top, m);
    s.low = __builtin_elementwise_min(s.low, m - (u16x2)(1));
}

template <int R>
__device__ __forceinline__ bool span_exact(const Span &s) {
    const uint32_t top = s.top.x > s.top.y ? s.top.x : s.top.y;
    const uint32_t low = (uint16_t)((s.low.x < s.low.y ? s.low.x : s.low.y) + 1);  // 0: no nonzero value
    const int e_top = (int)(top >> 7);
    const int e_low = (int)(low >> 7) > 1 ? (int)(low >> 7) : 1;
    return e_top - e_low <= kExactSpan<R>;
}

// The wide route's exact sum: S in two's complement in ten 32-bit words,
// bit 0 weighing 2^-133 (the smallest BF16 step).  16 values below 2^128 sum
// below 2^132, so 266 bits with the sign suffice.  The ranks are added one at
// a time, each as a piece of at most 40 bits carried (or borrowed) through
// the words above it: a short loop over few registers.
constexpr int kWideWords = 10;

__device__ __forceinline__ void wide_add(uint32_t (&w)[kWideWords], uint32_t bf16) {
    const uint32_t e = (bf16 >> 7) & 0xffu, f = bf16 & 0x7fu;
    const uint32_t mant = e ? (0x80u | f) : f;  // value = mant * 2^(pos - 133)
    const uint32_t pos = (e ? e : 1u) - 1u;
    const uint64_t piece = (uint64_t)mant << (pos & 31u);
    const uint32_t wi = pos >> 5, plo = (uint32_t)piece, phi = (uint32_t)(piece >> 32);
    const bool sub = (bf16 & 0x8000u) != 0;
    uint32_t carry = 0;  // carry when adding, borrow when subtracting
#pragma unroll
    for (int k = 0; k < kWideWords; ++k) {
        const uint32_t x = k == (int)wi ? plo : k == (int)wi + 1 ? phi : 0u;
        const uint64_t t = sub ? (uint64_t)w[k] - x - carry : (uint64_t)w[k] + x + carry;
        w[k] = (uint32_t)t;
        carry = (uint32_t)(t >> 32) & 1u;
    }
}

// The wide route for one element: rank r's BF16 pattern is g[r][i].
template <int R>
__device__ __forceinline__ float mean_wide(const uint16_t *const *g, int64_t i) {
    uint32_t w[kWideWords];
#pragma unroll
    for (int k = 0; k < kWideWords; ++k) w[k] = 0;
    bool finite = true;
    double s = 0.0;
#pragma unroll 1
    for (int r = 0; r < R; ++r) {
        const uint32_t v = g[r][i];
        finite &= (v & 0x7f80u) != 0x7f80u;
        s += (double)__uint_as_float(v << 16);
        if ((v & 0x7fffu) != 0) wide_add(w, v);
    }
    // NaN or an infinity: the IEEE result of the FP64 sum in rank order
    if (!finite) return mean_of<R>(s);
    const bool neg = (w[kWideWords - 1] >> 31) != 0;
    if (neg) {
        uint32_t c = 1;
#pragma unroll
        for (int k = 0; k < kWideWords; ++k) {
            const uint64_t t = (uint64_t)(~w[k]) + c;
            w[k] = (uint32_t)t;
            c = (uint32_t)(t >> 32);
        }
    }
    int top = -1;
#pragma unroll
    for (int k = 0; k < kWideWords; ++k)
        if (w[k]) top = k;
    if (top < 0) return 0.0f;
    // the top three words (zero below word 0) and whether any word under them is nonzero
    uint32_t hw = 0, mw = 0, lw = 0;
    bool below = false;
#pragma unroll
    for (int k = 0; k < kWideWords; ++k) {
        hw = k == top ? w[k] : hw;
        mw = k == top - 1 ? w[k] : mw;
        lw = k == top - 2 ? w[k] : lw;
        below |= (k < top - 2) && w[k] != 0;
    }
    const int sh = __builtin_clz(hw);
    uint64_t hi64 = ((uint64_t)hw << 32) | mw;
    uint32_t rest = lw;
    if (sh) {
        hi64 = (hi64 << sh) | (lw >> (32 - sh));
        rest = lw << sh;
    }
    uint64_t m53 = hi64 >> 11;
    if ((hi64 & 0x7ffu) != 0 || rest != 0 || below) m53 |= 1u;  // round to odd
    const double mag = ldexp((double)m53, 11 + 32 - sh + 32 * (top - 2) - 133);
    return mean_of<R>(neg ? -mag : mag);
}

// The wide route for element i of the R buffers g[r], and for the four
// elements from e0, loading their inputs again (only the rare lanes that
// fail span_exact take it).  Inlined: as a function call it gave every
// kernel a call stack in scratch memory, and the kernels with scratch ran
// three to four times slower (0.67 against 0.23 ms for the Qwen3-8B layer's
// norm pass), since scratch caps the waves in flight.  The ranks are added
// one at a time into ten words, so the route adds few registers.
template <int R>
__device__ __forceinline__ float mean_wide_at(const uint16_t *const *g, int64_t i) {
    return mean_wide<R>(g, i);
}

template <int R>
__device__ __forceinline__ float4 mean_wide_at4(const uint16_t *const *g, int64_t e0) {
    float4 o;
    o.x = mean_wide_at<R>(g, e0);
    o.y = mean_wide_at<R>(g, e0 + 1);
    o.z = mean_wide_at<R>(g, e0 + 2);
    o.w = mean_wide_at<R>(g, e0 + 3);
    return o;
}

// Fast route for the 2W elements held as BF16 in w[r][0..W-1] (two per word,
// the lower half first).  Returns false if the values fail span_exact: the
// caller must then take the wide route for them.
template <int R, int W>
__device__ __forceinline__ bool means_fast(const uint32_t (&w)[R][W], float (&g)[2 * W]) {
    Span sp = span_init();
#pragma unroll
    for (int j = 0; j < W; ++j) {
        double s_lo = 0.0, s_hi = 0.0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            s_lo += (double)bf16_lo(w[r][j]);
            s_hi += (double)bf16_hi(w[r][j]);
            if constexpr (R > 1) span_add(sp, w[r][j]);
        }
        g[2 * j] = mean_of<R>(s_lo);
        g[2 * j + 1] = mean_of<R>(s_hi);
    }
    if constexpr (R > 1) return span_exact<R>(sp);
    return true;
}

// g_bar of the 4 elements from e0 of the R buffers g[r], whose BF16 words
// (already loaded) are w.
template <int R>
__device__ __forceinline__ void mean4(const uint32_t (&w)[R][2], const uint16_t *const *g, int64_t e0,
                                      float (&out)[4]) {
    if (__builtin_expect(!means_fast<R, 2>(w, out), 0)) {
        const float4 t = mean_wide_at4<R>(g, e0);
        out[0] = t.x;
        out[1] = t.y;
        out[2] = t.z;
        out[3] = t.w;
    }
}

// g_bar of element i of the R buffers g[r].
template <int R>
__device__ __forceinline__ float mean1(const uint16_t *const *g, int64_t i) {
    uint32_t v[R];
    double s = 0.0;
    Span sp = span_init();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        v[r] = g[r][i];
        s += (double)__uint_as_float(v[r] << 16);
        span_add(sp, v[r]);
    }
    if constexpr (R > 1)
        if (!span_exact<R>(sp)) return mean_wide_at<R>(g, i);
    return mean_of<R>(s);
}

// Double-double accumulation.  S is the sum of the squares of FP32 values,
// each exact in FP64; it is carried as an unevaluated pair hi + lo (about
// 106 significant bits), so its final rounding to FP64 is that of the exact
// sum except when the exact sum lies within ~1e-28 of an FP64 rounding
// boundary.  two_sum is Knuth's error-free addition.
__device__ __forceinline__ void dd_add(double &hi, double &lo, double x) {
    const double s = hi + x;
    const double bb = s - hi;
    const double e = (hi - (s - bb)) + (x - bb);
    hi = s;
    lo += e;
}

__device__ __forceinline__ void dd_merge(double &hi, double &lo, double bhi, double blo) {
    const double s = hi + bhi;
    const double bb = s - hi;
    double e = (hi - (s - bb)) + (bhi - bb);
    e += lo + blo;
    hi = s + e;           // renormalised: hi is the pair rounded to FP64
    lo = e - (hi - s);
}

__device__ __forceinline__ void wave_merge(double &hi, double &lo) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const double oh = __shfl_xor(hi, off, 64);
        const double ol = __shfl_xor(lo, off, 64);
        dd_merge(hi, lo, oh, ol);
    }
}

// Block sum of one pair per thread in a fixed order: a fixed butterfly inside
// each wave, then the waves in index order.  Valid in thread 0.
template <int THREADS>
__device__ __forceinline__ void block_merge(double &hi, double &lo) {
    __shared__ double ws_hi[THREADS / 64], ws_lo[THREADS / 64];
    wave_merge(hi, lo);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        ws_hi[wave] = hi;
        ws_lo[wave] = lo;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        hi = ws_hi[0];
        lo = ws_lo[0];
#pragma unroll
        for (int k = 1; k < THREADS / 64; ++k) dd_merge(hi, lo, ws_hi[k], ws_lo[k]);
    }
}

// ---------------------------------------------------------------------------
// Norm partials: each tile is split into kNormSplit spans of kNormSpan
// elements, and block b sums g_bar^2 over span b of the segment (the grid is
// kNormSplit blocks per tile, those past the end write a zero pair).  Lanes
// read 4 elements per rank at a time (8-byte loads); when g_bar is stored,
// each lane's 4 FP32 results go out as one 16-byte store, contiguous across
// the wave.  Lane t handles the 4-element groups b*1024 + 256*j + t in
// increasing j; the read-only pass issues two groups before either is
// consumed, the pass that stores g_bar one (it runs under a residency cap,
// and more loads in flight per lane measured slower there).  Gradients and
// g_bar move with non-temporal loads and stores: they are not reused within
// the pass, and the 256 MB last-level cache cannot hold them until the
// update reads g_bar back.  The ragged tail of fewer than V
// elements is added by lane 0 of its span after the groups.  The per-lane
// order, the butterfly and the wave order are fixed, so a span's partial
// depends on its contents only.
__device__ __forceinline__ uint4 load_stream(const uint16_t *p) {
    const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(t.x, t.y, t.z, t.w);
}

template <int V>
__device__ __forceinline__ void load_stream_v(const uint16_t *p, uint32_t (&w)[V / 2]) {
    if constexpr (V == 8) {
        const u32x4 t = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
        w[0] = t.x; w[1] = t.y; w[2] = t.z; w[3] = t.w;
    } else {
        const u32x2 t = __builtin_nontemporal_load(reinterpret_cast<const u32x2 *>(p));
        w[0] = t.x; w[1] = t.y;
    }
}

template <int R, bool WRITE_GBAR>
__global__ __launch_bounds__(kNormThreads) void k_norm_partials(NormArgs a) {
    constexpr int V = 4;
    constexpr int kGroupsPerSpan = kNormSpan / V;
    constexpr int kUnroll = WRITE_GBAR ? 1 : 2;
    constexpr int kIters = kGroupsPerSpan / (kNormThreads * kUnroll);
    static_assert(kIters * kNormThreads * kUnroll == kGroupsPerSpan, "span must split evenly over the lanes");
    const int64_t n = a.n;
    const int64_t full_groups = n / V;
    const int64_t span0 = (int64_t)blockIdx.x * kGroupsPerSpan;
    double hi = 0.0, lo = 0.0;
    uint32_t wide = 0;  // bit (it * kUnroll + u): a group that takes the wide route
    for (int it = 0; it < kIters; ++it) {
        uint32_t raw[kUnroll][R][V / 2];
        bool ok[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int64_t q = span0 + (int64_t)(it * kUnroll + u) * kNormThreads + threadIdx.x;
            ok[u] = q < full_groups;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (ok[u]) {
                    load_stream_v<V>(a.g[r] + q * V, raw[u][r]);
                } else {
#pragma unroll
                    for (int w = 0; w < V / 2; ++w) raw[u][r][w] = 0;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            if (!ok[u]) continue;
            float g[V];
            if (__builtin_expect(!means_fast<R, V / 2>(raw[u], g), 0)) {
                wide |= 1u << (it * kUnroll + u);
                continue;
            }
#pragma unroll
            for (int e = 0; e < V; ++e) dd_add(hi, lo, (double)g[e] * (double)g[e]);
            if constexpr (WRITE_GBAR) {
                const int64_t e0 = (span0 + (int64_t)(it * kUnroll + u) * kNormThreads + threadIdx.x) * V;
                store_nt4(a.gbar_out + e0, make_float4(g[0], g[1], g[2], g[3]));
            }
        }
    }
    // the groups that failed the span check, in the same order, after the
    // loop, where the wide route's registers do not add to the loop's
    static_assert(kIters * kUnroll <= 32, "one bit per group of a lane");
    while (__builtin_expect(wide != 0, 0)) {
        const int k = __builtin_ctz(wide);
        wide &= wide - 1;
        const int64_t e0 = (span0 + (int64_t)k * kNormThreads + threadIdx.x) * V;
        const float4 t = mean_wide_at4<R>(a.g, e0);
        dd_add(hi, lo, (double)t.x * (double)t.x);
        dd_add(hi, lo, (double)t.y * (double)t.y);
        dd_add(hi, lo, (double)t.z * (double)t.z);
        dd_add(hi, lo, (double)t.w * (double)t.w);
        if constexpr (WRITE_GBAR) store_nt4(a.gbar_out + e0, t);
    }
    const int64_t tail0 = full_groups * V;
    if (threadIdx.x == 0 && tail0 < n && tail0 / kNormSpan == (int64_t)blockIdx.x) {
        for (int64_t i = tail0; i < n; ++i) {
            float g = mean1<R>(a.g, i);
            dd_add(hi, lo, (double)g * (double)g);
            if constexpr (WRITE_GBAR) a.gbar_out[i] = g;
        }
    }
    block_merge<kNormThreads>(hi, lo);
    if (threadIdx.x == 0) {
        a.partials[2 * blockIdx.x] = hi;
        a.partials[2 * blockIdx.x + 1] = lo;
    }
}

// First stage of the finalize for many pairs: block b merges the pairs
// b*kMergeRun + t + kMergeThreads*j (j = 0 .. 7) in increasing j per thread,
// then the threads by the fixed block tree, into merged pair b.  Pairs past
// the end count as zero.
__global__ __launch_bounds__(kMergeThreads) void k_norm_merge(const double *__restrict__ partials,
                                                              int64_t n_pairs, double *__restrict__ merged) {
    constexpr int kPer = kMergeRun / kMergeThreads;
    const double2 *pairs = reinterpret_cast<const double2 *>(partials);
    const int64_t base = (int64_t)blockIdx.x * kMergeRun + threadIdx.x;
    double2 b[kPer];
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
        const int64_t i = base + (int64_t)j * kMergeThreads;
        b[j] = i < n_pairs ? pairs[i] : make_double2(0.0, 0.0);
    }
    double hi = b[0].x, lo = b[0].y;
#pragma unroll
    for (int j = 1; j < kPer; ++j) dd_merge(hi, lo, b[j].x, b[j].y);
    block_merge<kMergeThreads>(hi, lo);
    if (threadIdx.x == 0) {
        merged[2 * blockIdx.x] = hi;
        merged[2 * blockIdx.x + 1] = lo;
    }
}

// One block: fixed-order sum of all span partials (pairs), then the norm, the
// clip coefficient and the non-finite flag.  Thread t takes the pairs
// t + 1024*j; pair j goes to the thread's accumulator j mod 4 (four
// independent chains), each merged in increasing j, and the four are then
// merged in order.  Loads are issued 16 at a time so that their latencies
// overlap.
__global__ __launch_bounds__(kFinalizeThreads) void k_norm_finalize(
    const double *__restrict__ partials, int64_t n_partials, double max_grad_norm,
    NormState *__restrict__ ns) {
    constexpr int kBatch = 16;
    constexpr int kChains = 4;
    const double2 *pairs = reinterpret_cast<const double2 *>(partials);
    double chi[kChains] = {0.0, 0.0, 0.0, 0.0}, clo[kChains] = {0.0, 0.0, 0.0, 0.0};
    for (int64_t i0 = threadIdx.x; i0 < n_partials; i0 += (int64_t)kBatch * kFinalizeThreads) {
        double2 b[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u) {
            const int64_t i = i0 + (int64_t)u * kFinalizeThreads;
            b[u] = i < n_partials ? pairs[i] : make_double2(0.0, 0.0);
        }
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
            if (i0 + (int64_t)u * kFinalizeThreads < n_partials) dd_merge(chi[u % kChains], clo[u % kChains], b[u].x, b[u].y);
    }
    double hi = chi[0], lo = clo[0];
#pragma unroll
    for (int c = 1; c < kChains; ++c) dd_merge(hi, lo, chi[c], clo[c]);
    block_merge<kFinalizeThreads>(hi, lo);
    if (threadIdx.x == 0) {
        const double S = hi;
        const double norm = sqrt(S);
        const int bad = !isfinite(S);
        double c = 1.0;
        if (max_grad_norm > 0.0 && !bad) {
            c = max_grad_norm / (norm + 1e-6);
            if (c > 1.0) c = 1.0;
        }
        ns->sumsq = S;
        ns->norm = norm;
        ns->clip = c;
        ns->nonfinite = bad;
        ns->pad = 0;
    }
}

// ---------------------------------------------------------------------------
// Fused update.

struct Consts {
    double c, lr_wd, beta1, omb1, beta2, omb2, step_size, inv_bc2, eps;
};

// p1, m' and v' are each rounded after every product and sum, in the order
// of their definition (no fused multiply-add).  m' cancels where b1*m is
// close to -(1-b1)*g -- common, since the inputs sit on the coarse BF16 grid
// -- and there a single-rounding fma and a two-rounding evaluation differ by
// a large relative amount of a result that is pure rounding noise.  Fixing
// the order makes m' (and v', p1) the same bits as the definition's.
__device__ __forceinline__ void moments(double pd, double md, double vd, double g, const Consts &k,
                                        double &p1, double &m1, double &v1) {
#pragma clang fp contract(off)
    p1 = pd - k.lr_wd * pd;
    m1 = k.beta1 * md + k.omb1 * g;
    v1 = k.beta2 * vd + k.omb2 * (g * g);
}

__device__ __forceinline__ void adamw(float &p, float &m, float &v, float g_bar, const Consts &k) {
#pragma clang fp contract(off)
    const double g = (double)g_bar * k.c;
    double p1, m1, v1;
    moments((double)p, (double)m, (double)v, g, k, p1, m1, v1);
    const double denom = sqrt(v1 * k.inv_bc2) + k.eps;
    const double pn = p1 - k.step_size * (m1 / denom);
    p = (float)pn;
    m = (float)m1;
    v = (float)v1;
}

// Lane t of the grid handles elements 4t .. 4t+3: each access of a wave is
// one contiguous run (1 KB of every FP32 array, 512 B of every BF16 one).
// Every load and store is non-temporal: under the residency cap this
// measured about 5% faster than plain accesses to the states and g_bar.
template <int R, bool CACHED>
__global__ __launch_bounds__(kUpdateThreads) void k_update(UpdateArgs a) {
    const NormState *ns = a.ns;
    if (ns->nonfinite) return;
    Consts k;
    k.c = ns->clip;
    k.lr_wd = a.lr_wd;
    k.beta1 = a.beta1;
    k.omb1 = a.one_minus_beta1;
    k.beta2 = a.beta2;
    k.omb2 = a.one_minus_beta2;
    k.step_size = a.step_size;
    k.inv_bc2 = a.inv_bc2;
    k.eps = a.eps;

    float *__restrict__ P = a.p;
    float *__restrict__ M = a.m;
    float *__restrict__ V = a.v;
    uint16_t *__restrict__ PB = a.pb;
    const float *__restrict__ GB = a.gbar;
    const int64_t n = a.n;
    const int64_t groups = n / kUpdVec;
    const int64_t gid = (int64_t)blockIdx.x * kUpdateThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kUpdateThreads;

    for (int64_t q = gid; q < groups; q += stride) {
        const int64_t e0 = q * kUpdVec;
        float g[kUpdVec];
        bool fast = true;
        if constexpr (CACHED) {
            const float4 a0 = load_nt4(GB + e0);
            g[0] = a0.x; g[1] = a0.y; g[2] = a0.z; g[3] = a0.w;
        } else {
            uint32_t raw[R][2];
            // read once: non-temporal, as in the norm pass
#pragma unroll
            for (int r = 0; r < R; ++r) load_stream_v<4>(a.g[r] + e0, raw[r]);
            fast = means_fast<R, 2>(raw, g);
        }
        float4 pv = load_nt4(P + e0);
        float4 mv = load_nt4(M + e0);
        float4 vv = load_nt4(V + e0);
        if (__builtin_expect(!fast, 0)) {
            // the wide route (see means_fast)
            const float4 t = mean_wide_at4<R>(a.g, e0);
            g[0] = t.x; g[1] = t.y; g[2] = t.z; g[3] = t.w;
        }
        float *pf = &pv.x, *mf = &mv.x, *vf = &vv.x;
#pragma unroll
        for (int e = 0; e < kUpdVec; ++e) adamw(pf[e], mf[e], vf[e], g[e], k);
        store_nt4(P + e0, pv);
        store_nt4(M + e0, mv);
        store_nt4(V + e0, vv);
        store_nt2(PB + e0, pack_bf16(pf[0], pf[1]), pack_bf16(pf[2], pf[3]));
    }
    // ragged tail of fewer than 4 elements
    if (gid == 0) {
        for (int64_t i = groups * kUpdVec; i < n; ++i) {
            float gb;
            if constexpr (CACHED) gb = GB[i];
            else gb = mean1<R>(a.g, i);
            float p = P[i], m = M[i], v = V[i];
            adamw(p, m, v, gb, k);
            P[i] = p; M[i] = m; V[i] = v;
            PB[i] = (uint16_t)bf16_rne(p);
        }
    }
}

// ---------------------------------------------------------------------------
// Measurement: the fused update's memory access pattern with trivial
// arithmetic (integer and FP32 adds instead of the FP64 AdamW), the same
// loads, stores, widths and lane mapping, from the R gradients or (CACHED)
// from stored g_bar.  Its rate is the ceiling that the update's own traffic
// mix allows on this part.  Overwrites the states.

template <int R, bool CACHED>
__global__ __launch_bounds__(kUpdateThreads) void k_update_pattern(UpdateArgs a) {
    float *__restrict__ P = a.p;
    float *__restrict__ M = a.m;
    float *__restrict__ V = a.v;
    uint16_t *__restrict__ PB = a.pb;
    const int64_t n = a.n;
    const int64_t groups = n / kUpdVec;
    const int64_t gid = (int64_t)blockIdx.x * kUpdateThreads + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * kUpdateThreads;
    for (int64_t q = gid; q < groups; q += stride) {
        const int64_t e0 = q * kUpdVec;
        uint32_t x = 0;
        if constexpr (CACHED) {
            const float4 t = load_nt4(a.gbar + e0);
            x = __float_as_uint(t.x) ^ __float_as_uint(t.y) ^ __float_as_uint(t.z) ^ __float_as_uint(t.w);
        } else {
#pragma unroll
            for (int r = 0; r < R; ++r) {
                uint32_t w[2];
                load_stream_v<4>(a.g[r] + e0, w);
                x ^= w[0] ^ w[1];
            }
        }
        const float gx = __uint_as_float((x & 0x007fffffu) | 0x3f800000u);
        float4 pv = load_nt4(P + e0), mv = load_nt4(M + e0), vv = load_nt4(V + e0);
        float *pf = &pv.x, *mf = &mv.x, *vf = &vv.x;
#pragma unroll
        for (int e = 0; e < kUpdVec; ++e) {
            pf[e] += gx;
            mf[e] += pf[e];
            vf[e] += mf[e];
        }
        store_nt4(P + e0, pv);
        store_nt4(M + e0, mv);
        store_nt4(V + e0, vv);
        store_nt2(PB + e0, (__float_as_uint(pf[0]) >> 16) | (__float_as_uint(pf[1]) & 0xffff0000u),
                  (__float_as_uint(pf[2]) >> 16) | (__float_as_uint(pf[3]) & 0xffff0000u));
    }
}

// ---------------------------------------------------------------------------
// Measurement: the g_bar-storing norm pass's memory access pattern with
// trivial arithmetic (xor of the ranks' bits instead of the exact mean and
// the double-double sum of squares): the same grid, lane mapping, loads,
// 16-byte stores and span pairs, under the same residency cap.  Its rate is
// the ceiling that the pass's own traffic mix allows on this part.  The
// ragged tail of fewer than 4 elements is left out.

template <int R>
__global__ __launch_bounds__(kNormThreads) void k_norm_pattern(NormArgs a) {
    constexpr int V = 4;
    constexpr int kGroupsPerSpan = kNormSpan / V;
    constexpr int kIters = kGroupsPerSpan / kNormThreads;
    const int64_t full_groups = a.n / V;
    const int64_t span0 = (int64_t)blockIdx.x * kGroupsPerSpan;
    uint32_t acc = 0;
    for (int it = 0; it < kIters; ++it) {
        const int64_t q = span0 + (int64_t)it * kNormThreads + threadIdx.x;
        if (q >= full_groups) break;
        uint32_t x0 = 0, x1 = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            uint32_t w[2];
            load_stream_v<V>(a.g[r] + q * V, w);
            x0 ^= w[0];
            x1 ^= w[1];
        }
        store_nt4(a.gbar_out + q * V, make_float4(bf16_lo(x0), bf16_hi(x0), bf16_lo(x1), bf16_hi(x1)));
        acc ^= x0 ^ x1;
    }
    double hi = (double)acc, lo = 0.0;
    block_merge<kNormThreads>(hi, lo);
    if (threadIdx.x == 0) {
        a.partials[2 * blockIdx.x] = hi;
        a.partials[2 * blockIdx.x + 1] = lo;
    }
}

// ---------------------------------------------------------------------------
// Mean gradient for the host-update route: g_bar of a chunk, FP32 or rounded
// to BF16, written to a staging slot that the copy engine then moves to host
// memory.  The rank gradients are read once and not reused (non-temporal).

template <int R, bool BF16>
__global__ __launch_bounds__(256) void k_gbar_out(GbarArgs a) {
    const int64_t n = a.n;
    const int64_t groups = n / kVec;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t q = gid; q < groups; q += stride) {
        uint32_t lo4[R][2], hi4[R][2];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint4 w = load_stream(a.g[r] + q * kVec);
            lo4[r][0] = w.x;
            lo4[r][1] = w.y;
            hi4[r][0] = w.z;
            hi4[r][1] = w.w;
        }
        float g[kVec], g4[4];
        mean4<R>(lo4, a.g, q * kVec, g4);
        g[0] = g4[0]; g[1] = g4[1]; g[2] = g4[2]; g[3] = g4[3];
        mean4<R>(hi4, a.g, q * kVec + 4, g4);
        g[4] = g4[0]; g[5] = g4[1]; g[6] = g4[2]; g[7] = g4[3];
        if constexpr (BF16) {
            uint4 b;
            b.x = pack_bf16(g[0], g[1]);
            b.y = pack_bf16(g[2], g[3]);
            b.z = pack_bf16(g[4], g[5]);
            b.w = pack_bf16(g[6], g[7]);
            reinterpret_cast<uint4 *>(a.out)[q] = b;
        } else {
            float4 *o = reinterpret_cast<float4 *>(a.out) + 2 * q;
            o[0] = make_float4(g[0], g[1], g[2], g[3]);
            o[1] = make_float4(g[4], g[5], g[6], g[7]);
        }
    }
    if (gid == 0) {
        for (int64_t i = groups * kVec; i < n; ++i) {
            const float g = mean1<R>(a.g, i);
            if constexpr (BF16) reinterpret_cast<uint16_t *>(a.out)[i] = (uint16_t)bf16_rne(g);
            else reinterpret_cast<float *>(a.out)[i] = g;
        }
    }
}

// ---------------------------------------------------------------------------
// Small helpers.

__global__ __launch_bounds__(256) void k_cast_bf16(const float *__restrict__ src,
                                                   uint16_t *__restrict__ dst, int64_t n) {
    const int64_t groups = n / kVec;
    const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t q = gid; q < groups; q += stride) {
        const float4 a0 = reinterpret_cast<const float4 *>(src + q * kVec)[0];
        const float4 a1 = reinterpret_cast<const float4 *>(src + q * kVec)[1];
        uint4 b;
        b.x = pack_bf16(a0.x, a0.y);
        b.y = pack_bf16(a0.z, a0.w);
        b.z = pack_bf16(a1.x, a1.y);
        b.w = pack_bf16(a1.z, a1.w);
        *reinterpret_cast<uint4 *>(dst + q * kVec) = b;
    }
    if (gid == 0)
        for (int64_t i = groups * kVec; i < n; ++i) dst[i] = (uint16_t)bf16_rne(src[i]);
}

__global__ __launch_bounds__(256) void k_copy16(uint4 *__restrict__ dst, const uint4 *__restrict__ src,
                                                int64_t n16) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += stride) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void k_fill_u32(uint32_t *__restrict__ dst, int64_t n_words, uint32_t value) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    const int64_t n4 = n_words / 4;
    uint4 v4 = make_uint4(value, value, value, value);
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride)
        reinterpret_cast<uint4 *>(dst)[i] = v4;
    if (blockIdx.x == 0 && threadIdx.x == 0)
        for (int64_t i = n4 * 4; i < n_words; ++i) dst[i] = value;
}

// ceil(a / b) for a >= 0, b > 0, without overflow near the int64 limit
inline int64_t cdiv(int64_t a, int64_t b) { return a / b + (a % b != 0); }

template <int R>
hipError_t norm_r(const NormArgs &a, int store_lds_pad, hipStream_t s) {
    const int64_t blocks = cdiv(a.n, kTile) * kNormSplit;
    if (a.gbar_out)
        hipLaunchKernelGGL((k_norm_partials<R, true>), dim3((uint32_t)blocks), dim3(kNormThreads), store_lds_pad, s,
                           a);
    else
        hipLaunchKernelGGL((k_norm_partials<R, false>), dim3((uint32_t)blocks), dim3(kNormThreads), 0, s, a);
    return hipGetLastError();
}

template <int R>
hipError_t update_r(const UpdateArgs &a, int64_t blocks, int lds_pad, hipStream_t s) {
    if (a.gbar)
        hipLaunchKernelGGL((k_update<1, true>), dim3((uint32_t)blocks), dim3(kUpdateThreads), lds_pad, s, a);
    else
        hipLaunchKernelGGL((k_update<R, false>), dim3((uint32_t)blocks), dim3(kUpdateThreads), lds_pad, s, a);
    return hipGetLastError();
}

template <int R>
hipError_t pattern_r(const UpdateArgs &a, int64_t blocks, int lds_pad, hipStream_t s) {
    if (a.gbar)
        hipLaunchKernelGGL((k_update_pattern<1, true>), dim3((uint32_t)blocks), dim3(kUpdateThreads), lds_pad, s, a);
    else
        hipLaunchKernelGGL((k_update_pattern<R, false>), dim3((uint32_t)blocks), dim3(kUpdateThreads), lds_pad, s, a);
    return hipGetLastError();
}

template <int R>
hipError_t norm_pattern_r(const NormArgs &a, int store_lds_pad, hipStream_t s) {
    const int64_t blocks = cdiv(a.n, kTile) * kNormSplit;
    hipLaunchKernelGGL((k_norm_pattern<R>), dim3((uint32_t)blocks), dim3(kNormThreads), store_lds_pad, s, a);
    return hipGetLastError();
}

template <int R>
hipError_t gbar_r(const GbarArgs &a, int64_t blocks, hipStream_t s) {
    if (a.bf16)
        hipLaunchKernelGGL((k_gbar_out<R, true>), dim3((uint32_t)blocks), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((k_gbar_out<R, false>), dim3((uint32_t)blocks), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace

#define SDP_FOR_EACH_R(X) X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16)

hipError_t launch_norm_partials(int R, const NormArgs &a, int store_lds_pad, hipStream_t s) {
    switch (R) {
#define CASE(r) case r: return norm_r<r>(a, store_lds_pad, s);
        SDP_FOR_EACH_R(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_norm_finalize(const double *partials, int64_t n_partials, double *merged, double max_grad_norm,
                                NormState *ns, hipStream_t s) {
    if (n_partials > kMergeRun) {
        if (!merged) return hipErrorInvalidValue;
        const int64_t blocks = cdiv(n_partials, kMergeRun);
        hipLaunchKernelGGL(k_norm_merge, dim3((uint32_t)blocks), dim3(kMergeThreads), 0, s, partials, n_partials,
                           merged);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        partials = merged;
        n_partials = blocks;
    }
    hipLaunchKernelGGL(k_norm_finalize, dim3(1), dim3(kFinalizeThreads), 0, s, partials, n_partials,
                       max_grad_norm, ns);
    return hipGetLastError();
}

hipError_t launch_update(int R, const UpdateArgs &a, int max_blocks, int lds_pad, hipStream_t s) {
    int64_t blocks = cdiv(a.n / kUpdVec, kUpdateThreads);
    if (blocks < 1) blocks = 1;
    if (max_blocks > 0 && blocks > max_blocks) blocks = max_blocks;
    switch (R) {
#define CASE(r) case r: return update_r<r>(a, blocks, lds_pad, s);
        SDP_FOR_EACH_R(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_update_pattern(int R, const UpdateArgs &a, int lds_pad, hipStream_t s) {
    int64_t blocks = cdiv(a.n / kUpdVec, kUpdateThreads);
    if (blocks < 1) blocks = 1;
    switch (R) {
#define CASE(r) case r: return pattern_r<r>(a, blocks, lds_pad, s);
        SDP_FOR_EACH_R(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_norm_pattern(int R, const NormArgs &a, int store_lds_pad, hipStream_t s) {
    switch (R) {
#define CASE(r) case r: return norm_pattern_r<r>(a, store_lds_pad, s);
        SDP_FOR_EACH_R(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gbar_out(int R, const GbarArgs &a, hipStream_t s) {
    int64_t blocks = cdiv(a.n / kVec, 256);
    if (blocks < 1) blocks = 1;
    if (blocks > 65536) blocks = 65536;
    switch (R) {
#define CASE(r) case r: return gbar_r<r>(a, blocks, s);
        SDP_FOR_EACH_R(CASE)
#undef CASE
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_cast_bf16(const float *src, uint16_t *dst, int64_t n, hipStream_t s) {
    int64_t blocks = cdiv(n / kVec, 256);
    if (blocks < 1) blocks = 1;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(k_cast_bf16, dim3((uint32_t)blocks), dim3(256), 0, s, src, dst, n);
    return hipGetLastError();
}

hipError_t launch_copy16(void *dst, const void *src, int64_t n16, int max_blocks, hipStream_t s) {
    int64_t blocks = cdiv(n16, 256);
    if (blocks < 1) blocks = 1;
    if (max_blocks > 0 && blocks > max_blocks) blocks = max_blocks;
    hipLaunchKernelGGL(k_copy16, dim3((uint32_t)blocks), dim3(256), 0, s, (uint4 *)dst,
                       (const uint4 *)src, n16);
    return hipGetLastError();
}

hipError_t launch_fill_u32(void *dst, int64_t n_words, uint32_t value, hipStream_t s) {
    int64_t blocks = cdiv(n_words / 4, 256);
    if (blocks < 1) blocks = 1;
    if (blocks > 16384) blocks = 16384;
    hipLaunchKernelGGL(k_fill_u32, dim3((uint32_t)blocks), dim3(256), 0, s, (uint32_t *)dst, n_words, value);
    return hipGetLastError();
}

}  // namespace sdp
