// AdamW on host cores for the host-update route: FP32 master weights and
// moments and BF16 parameters in host memory, fed the mean gradient that the
// GPU returned (FP32, or rounded to BF16 as in the paper's GPU-reduction
// route, Design, gradient return).
//
// Per element, in FP64, every product and sum rounded in the order written
// (this file is compiled with -ffp-contract=off, so nothing is fused):
//   g  = g_bar * c
//   p1 = p - (lr*wd) * p ;  m' = b1*m + (1-b1)*g ;  v' = b2*v + (1-b2)*(g*g)
//   p' = p1 - (lr/bc1) * (m' / (sqrt(v' * (1/bc2)) + eps))
// then one rounding of each state to FP32 and BF16 = round-to-nearest-even of
// the new FP32 master (NaN keeps sign and top payload bits, quiet bit set).
// These are the per-step constants and the order of operations of the fused
// GPU update.
//
// The AVX-512 path works on 8 elements per step, one FP64 lane each, so it
// performs exactly the scalar path's operations; the BF16 parameters leave
// with non-temporal stores (they are written once and read by the next
// parameter delivery, not by this core).
//
// Also here: the host lanes' BF16 rounding of FP32 values on its own
// (parameter delivery, and streamed mode with the BF16 parameters rounded on
// the host), integer round-to-nearest-even on the bit pattern, 16 values per
// AVX-512 step.
#include "sdp_host.h"

#include <immintrin.h>

#include <cmath>
#include <cstring>

namespace sdp_host {
namespace {

inline uint32_t bits_of(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    return u;
}

inline float float_of(uint32_t u) {
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

inline uint16_t bf16_rne(float f) {
    const uint32_t u = bits_of(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
    return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

inline float gbar_at(const AdamArgs &a, int64_t i) {
    if (a.gbar_bf16) return float_of((uint32_t)((const uint16_t *)a.gbar)[i] << 16);
    return ((const float *)a.gbar)[i];
}

inline void element(const AdamArgs &a, const AdamConsts &k, int64_t i) {
    const double g = (double)gbar_at(a, i) * k.c;
    const double p = a.p[i], m = a.m[i], v = a.v[i];
    const double p1 = p - k.lr_wd * p;
    const double m1 = k.beta1 * m + k.one_minus_beta1 * g;
    const double v1 = k.beta2 * v + k.one_minus_beta2 * (g * g);
    const double denom = std::sqrt(v1 * k.inv_bc2) + k.eps;
    const double pn = p1 - k.step_size * (m1 / denom);
    const float pf = (float)pn;
    a.p[i] = pf;
    a.m[i] = (float)m1;
    a.v[i] = (float)v1;
    a.pb[i] = bf16_rne(pf);
}

void range_scalar(const AdamArgs &a, const AdamConsts &k, int64_t i0, int64_t i1) {
    for (int64_t i = i0; i < i1; ++i) element(a, k, i);
}

__attribute__((target("avx512f,avx512bw,avx512vl,avx512dq"))) void range_avx512(const AdamArgs &a,
                                                                             const AdamConsts &k,
                                                                             int64_t i0, int64_t i1) {
    const __m512d c = _mm512_set1_pd(k.c);
    const __m512d lr_wd = _mm512_set1_pd(k.lr_wd);
    const __m512d b1 = _mm512_set1_pd(k.beta1), omb1 = _mm512_set1_pd(k.one_minus_beta1);
    const __m512d b2 = _mm512_set1_pd(k.beta2), omb2 = _mm512_set1_pd(k.one_minus_beta2);
    const __m512d step = _mm512_set1_pd(k.step_size), inv_bc2 = _mm512_set1_pd(k.inv_bc2);
    const __m512d eps = _mm512_set1_pd(k.eps);
    const __m256i abs_mask = _mm256_set1_epi32(0x7fffffff), inf = _mm256_set1_epi32(0x7f800000);
    const __m256i bias = _mm256_set1_epi32(0x7fff), one = _mm256_set1_epi32(1);
    const __m256i quiet = _mm256_set1_epi32(0x0040);
    const bool bf16_in = a.gbar_bf16 != 0;
    const uint16_t *gb16 = (const uint16_t *)a.gbar;
    const float *gf = (const float *)a.gbar;

    // scalar head up to a 16-byte boundary of the BF16 output, so that its
    // 16-byte stores are aligned
    int64_t i = i0;
    while (i < i1 && ((uintptr_t)(a.pb + i) & 15u) != 0) element(a, k, i++);
    for (; i + 8 <= i1; i += 8) {
        __m512d g;
        if (bf16_in) {
            const __m256i w = _mm256_cvtepu16_epi32(_mm_loadu_si128((const __m128i *)(gb16 + i)));
            g = _mm512_cvtps_pd(_mm256_castsi256_ps(_mm256_slli_epi32(w, 16)));
        } else {
            g = _mm512_cvtps_pd(_mm256_loadu_ps(gf + i));
        }
        g = _mm512_mul_pd(g, c);
        const __m512d p = _mm512_cvtps_pd(_mm256_loadu_ps(a.p + i));
        const __m512d m = _mm512_cvtps_pd(_mm256_loadu_ps(a.m + i));
        const __m512d v = _mm512_cvtps_pd(_mm256_loadu_ps(a.v + i));
        const __m512d p1 = _mm512_sub_pd(p, _mm512_mul_pd(lr_wd, p));
        const __m512d m1 = _mm512_add_pd(_mm512_mul_pd(b1, m), _mm512_mul_pd(omb1, g));
        const __m512d v1 = _mm512_add_pd(_mm512_mul_pd(b2, v), _mm512_mul_pd(omb2, _mm512_mul_pd(g, g)));
        const __m512d denom = _mm512_add_pd(_mm512_sqrt_pd(_mm512_mul_pd(v1, inv_bc2)), eps);
        const __m512d pn = _mm512_sub_pd(p1, _mm512_mul_pd(step, _mm512_div_pd(m1, denom)));
        const __m256 pf = _mm512_cvtpd_ps(pn);
        _mm256_storeu_ps(a.p + i, pf);
        _mm256_storeu_ps(a.m + i, _mm512_cvtpd_ps(m1));
        _mm256_storeu_ps(a.v + i, _mm512_cvtpd_ps(v1));
        // BF16 round to nearest even, NaN quieted
        const __m256i u = _mm256_castps_si256(pf);
        const __m256i hi = _mm256_srli_epi32(u, 16);
        const __m256i rne = _mm256_srli_epi32(_mm256_add_epi32(u, _mm256_add_epi32(bias, _mm256_and_si256(hi, one))), 16);
        const __mmask8 nan = _mm256_cmpgt_epu32_mask(_mm256_and_si256(u, abs_mask), inf);
        const __m256i b = _mm256_mask_blend_epi32(nan, rne, _mm256_or_si256(hi, quiet));
        _mm_stream_si128((__m128i *)(a.pb + i), _mm256_cvtepi32_epi16(b));
    }
    for (; i < i1; ++i) element(a, k, i);
    _mm_sfence();
}

uint16_t bf16_one(uint32_t x) {
    if ((x & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((x >> 16) | 0x0040u);
    return (uint16_t)((x + 0x7fffu + ((x >> 16) & 1u)) >> 16);
}

// Sixteen values per step: the same integer operations as bf16_one, the NaN
// case chosen by mask.  Finite values cannot carry out of 32 bits: the
// largest magnitude pattern plus the rounding bias stays below 2^32.
__attribute__((target("avx512f,avx512bw,avx512vl"))) void cast_avx512(const uint32_t *src, uint16_t *dst,
                                                                      int64_t n) {
    const __m512i abs_mask = _mm512_set1_epi32(0x7fffffff), inf = _mm512_set1_epi32(0x7f800000);
    const __m512i bias = _mm512_set1_epi32(0x7fff), one = _mm512_set1_epi32(1), quiet = _mm512_set1_epi32(0x40);
    int64_t i = 0;
    for (; i + 16 <= n; i += 16) {
        const __m512i x = _mm512_loadu_si512((const void *)(src + i));
        const __m512i hi = _mm512_srli_epi32(x, 16);
        const __m512i rne = _mm512_srli_epi32(_mm512_add_epi32(_mm512_add_epi32(x, bias), _mm512_and_si512(hi, one)), 16);
        const __mmask16 nan = _mm512_cmpgt_epu32_mask(_mm512_and_si512(x, abs_mask), inf);
        const __m512i r = _mm512_mask_blend_epi32(nan, rne, _mm512_or_si512(hi, quiet));
        _mm256_storeu_si256((__m256i *)(dst + i), _mm512_cvtepi32_epi16(r));
    }
    for (; i < n; ++i) dst[i] = bf16_one(src[i]);
}

}  // namespace

void cast_bf16(const float *src, uint16_t *dst, int64_t n) {
    const uint32_t *u = reinterpret_cast<const uint32_t *>(src);
    if (simd_best() >= kAvx512) {
        cast_avx512(u, dst, n);
        return;
    }
    for (int64_t i = 0; i < n; ++i) {
        uint32_t x;
        std::memcpy(&x, u + i, sizeof x);
        dst[i] = bf16_one(x);
    }
}

int simd_best() {
    static const int best = (__builtin_cpu_supports("avx512f") && __builtin_cpu_supports("avx512bw") &&
                             __builtin_cpu_supports("avx512vl") && __builtin_cpu_supports("avx512dq"))
                                ? kAvx512
                                : kScalar;
    return best;
}

void adamw_range(const AdamArgs &a, const AdamConsts &k, int64_t i0, int64_t i1, int simd) {
    if (i1 <= i0) return;
    // round to nearest even, all exceptions masked, no flush-to-zero or
    // denormals-are-zero, whatever the calling thread had set
    const unsigned saved = _mm_getcsr();
    _mm_setcsr(0x1f80u);
    if (simd >= kAvx512 && simd_best() >= kAvx512)
        range_avx512(a, k, i0, i1);
    else
        range_scalar(a, k, i0, i1);
    _mm_setcsr(saved);
}

}  // namespace sdp_host
