/* Element-wise comparison of GPU results with the oracle's (test helper).
 * Plain loops under OpenMP; no arithmetic of the update itself. */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* FP32: worst relative error over elements whose reference is finite and
 * non-zero, count of elements where the reference is zero but the result is
 * not, count where finiteness differs, count of identical bit patterns. */
void pc_compare_f32(const float *got, const float *ref, int64_t n, double *max_rel,
                    int64_t *worst_idx, int64_t *zero_mismatch, int64_t *finite_mismatch,
                    int64_t *bit_equal)
{
    double worst = 0.0;
    int64_t wi = -1, zm = 0, fm = 0, be = 0;
#pragma omp parallel
    {
        double lw = 0.0;
        int64_t lwi = -1, lzm = 0, lfm = 0, lbe = 0;
#pragma omp for schedule(static) nowait
        for (int64_t i = 0; i < n; ++i) {
            uint32_t a, b;
            memcpy(&a, &got[i], 4);
            memcpy(&b, &ref[i], 4);
            lbe += a == b;
            double g = got[i], r = ref[i];
            int fg = isfinite(g), fr = isfinite(r);
            if (fg != fr) { ++lfm; continue; }
            if (!fr) continue;
            if (r == 0.0) { lzm += g != 0.0; continue; }
            double rel = fabs(g - r) / fabs(r);
            if (rel > lw) { lw = rel; lwi = i; }
        }
#pragma omp critical
        {
            if (lw > worst) { worst = lw; wi = lwi; }
            zm += lzm; fm += lfm; be += lbe;
        }
    }
    *max_rel = worst;
    *worst_idx = wi;
    *zero_mismatch = zm;
    *finite_mismatch = fm;
    *bit_equal = be;
}

/* BF16 codes: number that differ, number whose sign differs, number that
 * differ by more than one in the magnitude code. */
void pc_compare_bf16(const uint16_t *got, const uint16_t *ref, int64_t n, int64_t *n_diff,
                     int64_t *n_sign, int64_t *n_far)
{
    int64_t d = 0, s = 0, f = 0;
#pragma omp parallel for schedule(static) reduction(+ : d, s, f)
    for (int64_t i = 0; i < n; ++i) {
        if (got[i] == ref[i]) continue;
        ++d;
        if ((got[i] >> 15) != (ref[i] >> 15)) ++s;
        int dm = (int)(got[i] & 0x7fff) - (int)(ref[i] & 0x7fff);
        if (dm > 1 || dm < -1) ++f;
    }
    *n_diff = d;
    *n_sign = s;
    *n_far = f;
}

/* Bitwise equality of two byte ranges, in parallel. */
int pc_equal(const uint8_t *a, const uint8_t *b, int64_t n)
{
    int64_t bad = 0;
#pragma omp parallel for schedule(static) reduction(+ : bad)
    for (int64_t i = 0; i < n; i += 4096) {
        int64_t len = n - i < 4096 ? n - i : 4096;
        bad += memcmp(a + i, b + i, (size_t)len) != 0;
    }
    return bad == 0;
}
