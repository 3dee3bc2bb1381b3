/*
 * Seeded synthetic inputs for the aggregate + clip + AdamW + BF16 path.
 *
 * This file produces input values only: FP32 normal draws, optional outlier
 * scaling, and seeds.  It holds none of the update's arithmetic (no mean, no
 * norm, no AdamW, no BF16 rounding); gradients are rounded to BF16 by the
 * caller with a library cast.  Both the CPU oracle and the HIP path consume
 * what it writes.
 *
 * Generator: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), written from that paper's definition:
 * a 4x32-bit counter, a 2x32-bit key, ten rounds of two 32x32->64 multiplies
 * whose high halves are xored with the other counter words and the key, the
 * key bumped by two Weyl constants between rounds.  Normals come from the
 * Box-Muller transform of two uniforms.  Element i of a stream uses counter
 * block i >> 1; even i takes the cosine branch and the third output word as
 * its outlier uniform, odd i the sine branch and the fourth word.  Every value
 * therefore depends on (seed, i) only, so any slice regenerates bit-identically
 * whatever the thread count.
 *
 * Seeds are derived with the splitmix64 mixer (Steele, Lea, Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA'14).
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox_round(uint32_t c[4], uint32_t k0, uint32_t k1)
{
    uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
    uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c[1] ^ k0;
    uint32_t n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
}

/* Philox4x32-10 of counter (ctr_lo, ctr_hi, 0, 0) under a 64-bit key. */
void synth_philox4x32_10(uint64_t key, uint64_t ctr, uint32_t out[4])
{
    uint32_t c[4] = {(uint32_t)ctr, (uint32_t)(ctr >> 32), 0u, 0u};
    uint32_t k0 = (uint32_t)key, k1 = (uint32_t)(key >> 32);
    for (int r = 0; r < 10; ++r) {
        philox_round(c, k0, k1);
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = c[0];
    out[1] = c[1];
    out[2] = c[2];
    out[3] = c[3];
}

uint64_t synth_splitmix64(uint64_t x)
{
    uint64_t z = x + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Seed of one stream: a splitmix64 chain over the fields that name it. */
uint64_t synth_seed(const int64_t *fields, int n_fields)
{
    uint64_t h = 0x5D9D9ull;
    for (int i = 0; i < n_fields; ++i)
        h = synth_splitmix64(h ^ (uint64_t)fields[i]);
    return h;
}

/* Uniform on the open interval (0, 1) from 32 random bits. */
static inline double u01(uint32_t x)
{
    return ((double)x + 0.5) * (1.0 / 4294967296.0);
}

static const double TWO_PI = 6.283185307179586476925286766559;

/* Standard normal and outlier uniform of element i of stream `seed`. */
static inline void draw(uint64_t seed, int64_t i, double *z, double *u_out)
{
    uint32_t w[4];
    synth_philox4x32_10(seed, (uint64_t)i >> 1, w);
    double r = sqrt(-2.0 * log(u01(w[0])));
    double th = TWO_PI * u01(w[1]);
    if ((i & 1) == 0) {
        *z = r * cos(th);
        *u_out = u01(w[2]);
    } else {
        *z = r * sin(th);
        *u_out = u01(w[3]);
    }
}

/* Both normals and both outlier uniforms of counter block j (elements 2j
 * and 2j+1); the same values draw() gives element by element. */
static inline void draw_pair(uint64_t seed, int64_t j, double z[2], double u[2])
{
    uint32_t w[4];
    synth_philox4x32_10(seed, (uint64_t)j, w);
    double r = sqrt(-2.0 * log(u01(w[0])));
    double th = TWO_PI * u01(w[1]);
    z[0] = r * cos(th);
    z[1] = r * sin(th);
    u[0] = u01(w[2]);
    u[1] = u01(w[3]);
}

static inline float scaled(double z, double u, double sigma, double outlier_p,
                           double outlier_scale)
{
    double x = sigma * z;
    if (outlier_p > 0.0 && u < outlier_p)
        x *= outlier_scale;
    return (float)x;
}

/*
 * out[k] = (float)(sigma * z(start + k)) for k in [0, n), where z is the
 * stream's standard normal; when outlier_p > 0 the value is first multiplied
 * by outlier_scale wherever that element's outlier uniform is below
 * outlier_p.  Parallel over counter blocks; the result does not depend on
 * the number of threads.
 */
void synth_normal_f32(uint64_t seed, int64_t start, int64_t n, double sigma,
                      double outlier_p, double outlier_scale, float *out)
{
    if (n <= 0)
        return;
    int64_t end = start + n;
    int64_t j0 = start >> 1, j1 = (end + 1) >> 1;
#pragma omp parallel for schedule(static)
    for (int64_t j = j0; j < j1; ++j) {
        double z[2], u[2];
        draw_pair(seed, j, z, u);
        for (int h = 0; h < 2; ++h) {
            int64_t i = 2 * j + h;
            if (i >= start && i < end)
                out[i - start] = scaled(z[h], u[h], sigma, outlier_p, outlier_scale);
        }
    }
}

/* Same values as synth_normal_f32, at an arbitrary list of element indices. */
void synth_normal_f32_at(uint64_t seed, const int64_t *idx, int64_t n,
                         double sigma, double outlier_p, double outlier_scale,
                         float *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t k = 0; k < n; ++k) {
        double z, u;
        draw(seed, idx[k], &z, &u);
        double x = sigma * z;
        if (outlier_p > 0.0 && u < outlier_p)
            x *= outlier_scale;
        out[k] = (float)x;
    }
}

/* Raw 32-bit words of consecutive counter blocks, for statistical tests. */
void synth_raw_u32(uint64_t seed, int64_t start_block, int64_t n_blocks,
                   uint32_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t b = 0; b < n_blocks; ++b)
        synth_philox4x32_10(seed, (uint64_t)(start_block + b), out + 4 * b);
}
