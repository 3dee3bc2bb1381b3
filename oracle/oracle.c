/*
 * CPU oracle of the data-parallel update -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg load
 * this file's library.  The HIP library never includes or calls it and the
 * two share no code.
 *
 * What it computes, per call over a list of flat layer segments that all have
 * R gradient buffers:
 *   1. g_bar[i] = fp32( (exact sum over ranks r of bf16 G_r[i]) / R ),
 *      rounded once -- the rank gradients are summed and averaged into one
 *      gradient (Design, shared host state and communication routes:
 *      gradient return by GPU reduction).
 *   2. S = sum over every element of every segment of g_bar[i]^2, the
 *      exact sum rounded once to FP64; norm = sqrt(S).  The paper never
 *      mentions clipping; the global L2 norm of the mean gradient is taken
 *      as the quantity to clip by.
 *   3. c = min(1, max_norm / (norm + 1e-6)) when max_norm > 0, else 1.
 *      A non-finite norm leaves every state unchanged.
 *   4. AdamW per element in FP64 (Loshchilov & Hutter, decoupled weight
 *      decay; Kingma & Ba bias correction), with g = g_bar[i] * c:
 *        p1 = p - (lr * wd) * p
 *        m' = beta1 * m + (1 - beta1) * g
 *        v' = beta2 * v + (1 - beta2) * g^2
 *        p' = p1 - lr * (m' / (1 - beta1^t)) / (sqrt(v' / (1 - beta2^t)) + eps)
 *      The paper calls the update mixed-precision Adam over FP32 master
 *      weights and FP32 moments (Background, training states table; Design,
 *      the rank-0 update worker).
 *   5. master = fp32(p'), exp_avg = fp32(m'), exp_avg_sq = fp32(v'),
 *      param_bf16 = bf16(master) -- BF16 compute weights for the next
 *      dispatch (training states table; Design, overlap within a layer).
 * Variant for a mean gradient returned to the host in BF16 (the paper's
 * GPU-reduction route hands one BF16 gradient to the host update; Design,
 * gradient return, and the per-layer reduce -> D2H -> Adam chain): step 4
 * then takes g = bf16(g_bar[i]) * c, while steps 2 and 3 still use the FP32
 * g_bar, so the clip decision does not depend on the transport format.
 * fp32() is the C conversion from double (round to nearest, ties to even);
 * bf16() is round to nearest even on the 8-bit significand, written below
 * from that definition.
 *
 * Parallelism: the per-element loops (independent elements) run under
 * OpenMP; the norm's exact sum is split over threads and merged exactly.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double f32_bits_value(uint32_t bits)
{
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* Round an FP32 value to the nearest BF16 value, ties to the BF16 value
 * whose last significand bit is zero.  BF16 keeps the FP32 sign and exponent
 * and the top 7 stored significand bits, so its values are exactly the FP32
 * values whose low 16 bits are zero.  The two candidates are the truncation
 * of |x| and the next BF16 value above it; an FP32 value above the largest
 * finite BF16 value by half a BF16 step or more rounds to infinity.  NaN
 * stays NaN with the quiet bit set; infinities and signed zeros are kept;
 * subnormals are rounded like any other value. */
uint16_t orc_bf16_from_f32(float x)
{
    uint32_t u;
    memcpy(&u, &x, sizeof u);
    uint32_t sign = u & 0x80000000u;
    uint32_t mag = u & 0x7fffffffu;
    if (mag > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t lo = mag & 0xffff0000u;
    if (lo == mag)
        return (uint16_t)(u >> 16);
    uint32_t hi = lo + 0x10000u;
    double a = f32_bits_value(mag);
    double vlo = f32_bits_value(lo);
    /* one step above the largest finite BF16 magnitude is 2^128 */
    double vhi = (hi == 0x7f800000u) ? ldexp(1.0, 128) : f32_bits_value(hi);
    double dlo = a - vlo, dhi = vhi - a;
    uint32_t pick;
    if (dlo < dhi)
        pick = lo;
    else if (dhi < dlo)
        pick = hi;
    else
        pick = ((lo >> 16) & 1u) ? hi : lo;
    return (uint16_t)((sign | pick) >> 16);
}

float orc_f32_from_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

void orc_bf16_array(const float *x, uint16_t *out, int64_t n)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = orc_bf16_from_f32(x[i]);
}

/* Step 1: the mean over ranks of one element's gradients, rounded once to
 * FP32: g_bar = fp32(S / R), where S is the exact sum of the R BF16 values
 * (Design, gradient return by GPU reduction: the reduction sums the ranks'
 * gradients and averages them).  A sum that is exactly zero gives +0.
 * If any value is an infinity or a NaN the mean is the IEEE result of the
 * FP64 sum in rank order divided by R (NaN or an infinity; the norm is then
 * not finite and no state changes).
 *
 * Two routes, both giving that one rounding:
 *  - when R is a power of two and every addition of the FP64 sum in rank
 *    order is exact (each TwoSum error term is zero), S is that FP64 sum and
 *    S / R is exact in FP64, so its conversion to FP32 is the only rounding;
 *  - otherwise S is formed exactly as a fixed-point integer, divided by R
 *    with a remainder, and the quotient is rounded to FP32 by hand. */

/* Unsigned fixed-point integer of MEAN_LIMBS little-endian 64-bit limbs whose
 * bit 0 has weight 2^MEAN_E0.  A BF16 value is M * 2^(k) with an integer
 * M < 2^8 and k >= -133; at most ORC_MAX_RANKS (2^6) of them, each below
 * 2^128, sum below 2^134, so 134 - MEAN_E0 = 287 bits suffice.  The 20 bits
 * below 2^-133 hold the quotient's bits down to 2^-153, under the FP32
 * rounding position of the smallest subnormal (2^-149). */
#define MEAN_E0 (-153)
#define MEAN_LIMBS 5
typedef struct {
    uint64_t w[MEAN_LIMBS];
} orc_fix;

static void fix_add_at(orc_fix *a, int k, uint64_t v)
{
    while (v != 0 && k < MEAN_LIMBS) {
        uint64_t old = a->w[k];
        a->w[k] = old + v;
        v = a->w[k] < old; /* carry */
        ++k;
    }
}

/* a += m * 2^b (b >= 0, m < 2^8). */
static void fix_add_shifted(orc_fix *a, uint64_t m, int b)
{
    int k = b >> 6, s = b & 63;
    fix_add_at(a, k, m << s);
    if (s > 56)
        fix_add_at(a, k + 1, m >> (64 - s));
}

static int fix_cmp(const orc_fix *a, const orc_fix *b)
{
    for (int k = MEAN_LIMBS - 1; k >= 0; --k)
        if (a->w[k] != b->w[k])
            return a->w[k] < b->w[k] ? -1 : 1;
    return 0;
}

/* a -= b, for a >= b. */
static void fix_sub(orc_fix *a, const orc_fix *b)
{
    uint64_t borrow = 0;
    for (int k = 0; k < MEAN_LIMBS; ++k) {
        uint64_t x = a->w[k], y = b->w[k];
        uint64_t d = x - y - borrow;
        borrow = (x < y) || (x == y && borrow);
        a->w[k] = d;
    }
}

/* a = floor(a / d); returns a mod d (schoolbook division by one word). */
static uint64_t fix_div_small(orc_fix *a, uint32_t d)
{
    unsigned __int128 rem = 0;
    for (int k = MEAN_LIMBS - 1; k >= 0; --k) {
        unsigned __int128 cur = (rem << 64) | a->w[k];
        a->w[k] = (uint64_t)(cur / d);
        rem = cur % d;
    }
    return (uint64_t)rem;
}

static int fix_msb(const orc_fix *a) /* -1 for zero */
{
    for (int k = MEAN_LIMBS - 1; k >= 0; --k)
        if (a->w[k])
            return k * 64 + 63 - __builtin_clzll(a->w[k]);
    return -1;
}

static int fix_bit(const orc_fix *a, int pos)
{
    return pos >= 0 ? (int)((a->w[pos >> 6] >> (pos & 63)) & 1u) : 0;
}

static int fix_any_below(const orc_fix *a, int pos) /* any bit at index < pos */
{
    if (pos <= 0)
        return 0;
    int k = pos >> 6, s = pos & 63;
    for (int j = 0; j < k; ++j)
        if (a->w[j])
            return 1;
    return s ? (a->w[k] & ((1ull << s) - 1)) != 0 : 0;
}

/* fp32(S / R) for finite BF16 values, through the exact integer S. */
static float mean_exact(const uint16_t *const *grads, int32_t R, int64_t i)
{
    orc_fix pos, neg;
    memset(&pos, 0, sizeof pos);
    memset(&neg, 0, sizeof neg);
    for (int32_t r = 0; r < R; ++r) {
        uint16_t b = grads[r][i];
        uint32_t e = (b >> 7) & 0xffu, f = b & 0x7fu;
        /* value = M * 2^(k): normal M = 1.f (8 bits), k = e - 127 - 7;
         * subnormal M = 0.f, k = 1 - 127 - 7 */
        uint64_t M = e ? (0x80u | f) : f;
        int k = (e ? (int)e : 1) - 134;
        fix_add_shifted((b & 0x8000u) ? &neg : &pos, M, k - MEAN_E0);
    }
    int sign = 0;
    if (fix_cmp(&pos, &neg) >= 0) {
        fix_sub(&pos, &neg);
    } else {
        fix_sub(&neg, &pos);
        pos = neg;
        sign = 1;
    }
    uint64_t rem = fix_div_small(&pos, (uint32_t)R);
    int msb = fix_msb(&pos);
    if (msb < 0)
        return 0.0f; /* S = 0 (a nonzero S is at least 2^-133, its quotient at least 2^-139) */
    /* keep 24 significant bits, or fewer below 2^-126, where the FP32 grid
     * is fixed at 2^-149 */
    int lsb = msb + MEAN_E0 >= -126 ? msb - 23 : -149 - MEAN_E0;
    uint64_t mant = 0;
    for (int q = msb; q >= lsb; --q)
        mant = (mant << 1) | (uint64_t)fix_bit(&pos, q);
    int round = fix_bit(&pos, lsb - 1);
    int sticky = rem != 0 || fix_any_below(&pos, lsb - 1);
    if (round && (sticky || (mant & 1u)))
        ++mant; /* may become 2^24 (or 2^23 below 2^-126): still exact */
    double mag = ldexp((double)mant, lsb + MEAN_E0);
    return (float)(sign ? -mag : mag); /* exact: mag is an FP32 value */
}

float orc_mean_grad(const uint16_t *const *grads, int32_t R, int64_t i)
{
    double s = 0.0;
    int exact = 1, finite = 1;
    for (int32_t r = 0; r < R; ++r) {
        double x = (double)orc_f32_from_bf16(grads[r][i]);
        if (!isfinite(x))
            finite = 0;
        /* TwoSum (Knuth): t + err = s + x exactly */
        double t = s + x;
        double xv = t - s;
        double err = (s - (t - xv)) + (x - xv);
        if (err != 0.0)
            exact = 0;
        s = t;
    }
    if (!finite)
        return (float)(s / (double)R);
    if (exact && (R & (R - 1)) == 0)
        return (float)(s / (double)R);
    return mean_exact(grads, R, i);
}

void orc_mean_grads(const uint16_t *const *grads, int32_t R, int64_t n, float *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = orc_mean_grad(grads, R, i);
}

/* Exact summation.  S is defined as the exact sum of the squares rounded
 * once to FP64.  Each square of an FP32 value is exact in FP64, so the sum
 * is accumulated without rounding in a fixed-point integer whose bit 0 has
 * weight 2^ACC_E0 (ACC_LIMBS little-endian 64-bit limbs: every finite
 * double, plus 64 bits of headroom for carries), then rounded to nearest,
 * ties to even.  Being exact, the sum does not depend on the order or
 * grouping of its terms, so threads may each accumulate a share. */
#define ACC_E0 (-1074)
#define ACC_LIMBS 35
typedef struct {
    uint64_t limb[ACC_LIMBS];
} orc_acc;

static void acc_add_at(orc_acc *a, int k, uint64_t v)
{
    while (v != 0 && k < ACC_LIMBS) {
        uint64_t old = a->limb[k];
        a->limb[k] = old + v;
        v = a->limb[k] < old; /* carry */
        ++k;
    }
}

/* Add a finite x >= 0. */
static void acc_add(orc_acc *a, double x)
{
    uint64_t bits;
    memcpy(&bits, &x, sizeof bits);
    uint64_t e = (bits >> 52) & 0x7ff;
    uint64_t m = bits & ((1ull << 52) - 1);
    if (e == 0 && m == 0)
        return;
    int b; /* weight of m's least bit is 2^(b + ACC_E0) */
    if (e == 0) {
        b = 0; /* subnormal: m * 2^-1074 */
    } else {
        m |= 1ull << 52;
        b = (int)e - 1075 - ACC_E0;
    }
    int k = b >> 6, s = b & 63;
    acc_add_at(a, k, m << s);
    if (s != 0)
        acc_add_at(a, k + 1, m >> (64 - s));
}

static void acc_merge(orc_acc *a, const orc_acc *b)
{
    for (int k = 0; k < ACC_LIMBS; ++k)
        acc_add_at(a, k, b->limb[k]);
}

static int acc_bit(const orc_acc *a, int pos)
{
    return pos >= 0 ? (int)((a->limb[pos >> 6] >> (pos & 63)) & 1u) : 0;
}

static int acc_any_below(const orc_acc *a, int pos) /* any bit at index < pos */
{
    if (pos <= 0)
        return 0;
    int k = pos >> 6, s = pos & 63;
    for (int j = 0; j < k; ++j)
        if (a->limb[j])
            return 1;
    return s ? (a->limb[k] & ((1ull << s) - 1)) != 0 : 0;
}

/* Round the accumulated value to the nearest double, ties to even.  (The
 * values summed here are at least 2^-298, so the result is never in the
 * subnormal range, where ldexp would round a second time.) */
static double acc_round(const orc_acc *a)
{
    int top = ACC_LIMBS - 1;
    while (top >= 0 && a->limb[top] == 0)
        --top;
    if (top < 0)
        return 0.0;
    int msb = top * 64 + 63 - __builtin_clzll(a->limb[top]);
    int lsb = msb - 52; /* lowest bit kept in a 53-bit significand */
    uint64_t mant = 0;
    for (int pos = msb; pos >= lsb; --pos)
        mant = (mant << 1) | (uint64_t)acc_bit(a, pos);
    if (acc_bit(a, lsb - 1) && (acc_any_below(a, lsb - 1) || (mant & 1u)))
        ++mant; /* may become 2^53, still exact */
    return ldexp((double)mant, lsb + ACC_E0);
}

/* Correctly rounded sum of x[i]^2 (test hook for the exact summation). */
double orc_sum_squares_f32(const float *x, int64_t n)
{
    orc_acc total;
    memset(&total, 0, sizeof total);
    double special = 0.0; /* non-finite terms propagate as in IEEE addition */
#pragma omp parallel
    {
        orc_acc mine;
        memset(&mine, 0, sizeof mine);
        double sp = 0.0;
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            double g = (double)x[i];
            double t = g * g;
            if (isfinite(t))
                acc_add(&mine, t);
            else
                sp += t;
        }
#pragma omp critical
        {
            acc_merge(&total, &mine);
            special += sp;
        }
    }
    if (special != 0.0 || isnan(special))
        return special;
    return acc_round(&total);
}

/* Step 2: global L2 norm of the mean gradient over all segments:
 * sqrt of the exactly rounded sum of g_bar^2 over every element. */
double orc_grad_norm(const orc_segment *segs, int32_t n_segs, int32_t R)
{
    orc_acc total;
    memset(&total, 0, sizeof total);
    double special = 0.0;
    for (int32_t s = 0; s < n_segs; ++s) {
        const uint16_t *const *g = segs[s].grads;
        const int64_t n = segs[s].numel;
#pragma omp parallel
        {
            orc_acc mine;
            memset(&mine, 0, sizeof mine);
            double sp = 0.0;
#pragma omp for schedule(static)
            for (int64_t i = 0; i < n; ++i) {
                double gb = (double)orc_mean_grad(g, R, i);
                double t = gb * gb;
                if (isfinite(t))
                    acc_add(&mine, t);
                else
                    sp += t;
            }
#pragma omp critical
            {
                acc_merge(&total, &mine);
                special += sp;
            }
        }
    }
    if (special != 0.0 || isnan(special))
        return sqrt(special);
    return sqrt(acc_round(&total));
}

/* Step 3: clip coefficient. */
double orc_clip_coef(double norm, double max_grad_norm)
{
    if (!(max_grad_norm > 0.0))
        return 1.0;
    double c = max_grad_norm / (norm + 1e-6);
    return c < 1.0 ? c : 1.0;
}

/* Step 4 for one element, no rounding. */
static void adamw_element(double p, double m, double v, double g,
                          const orc_hparams *hp, double bc1, double bc2,
                          double *po, double *mo, double *vo)
{
    double p1 = p - (hp->lr * hp->weight_decay) * p;
    double m1 = hp->beta1 * m + (1.0 - hp->beta1) * g;
    double v1 = hp->beta2 * v + (1.0 - hp->beta2) * (g * g);
    double m_hat = m1 / bc1;
    double v_hat = v1 / bc2;
    *po = p1 - hp->lr * m_hat / (sqrt(v_hat) + hp->eps);
    *mo = m1;
    *vo = v1;
}

static void bias_corrections(const orc_hparams *hp, double *bc1, double *bc2)
{
    *bc1 = 1.0 - pow(hp->beta1, (double)hp->step);
    *bc2 = 1.0 - pow(hp->beta2, (double)hp->step);
}

/* Step 4 on FP64 arrays with FP64 results (used by the library cross-check). */
void orc_adamw_f64(int64_t n, const double *p, const double *m, const double *v,
                   const double *g, const orc_hparams *hp,
                   double *p_out, double *m_out, double *v_out)
{
    double bc1, bc2;
    bias_corrections(hp, &bc1, &bc2);
    for (int64_t i = 0; i < n; ++i)
        adamw_element(p[i], m[i], v[i], g[i], hp, bc1, bc2,
                      &p_out[i], &m_out[i], &v_out[i]);
}

/* Steps 4 and 5 for one element given its mean gradient and clip coefficient. */
static void update_one(float *p, float *m, float *v, uint16_t *pb, float g_bar,
                       double c, const orc_hparams *hp, double bc1, double bc2)
{
    double po, mo, vo;
    adamw_element((double)*p, (double)*m, (double)*v, (double)g_bar * c, hp,
                  bc1, bc2, &po, &mo, &vo);
    *p = (float)po;
    *m = (float)mo;
    *v = (float)vo;
    *pb = orc_bf16_from_f32(*p);
}

/* The gradient step 4 consumes: g_bar, or g_bar rounded to BF16. */
static float update_gradient(float g_bar, int gbar_bf16)
{
    return gbar_bf16 ? orc_f32_from_bf16(orc_bf16_from_f32(g_bar)) : g_bar;
}

/* One full optimizer step over all segments; states are updated in place.
 * Returns ORC_NONFINITE (states untouched) when the norm is not finite. */
int orc_step(orc_segment *segs, int32_t n_segs, int32_t R, const orc_hparams *hp,
             double *norm_out)
{
    return orc_step_fmt(segs, n_segs, R, hp, 0, norm_out);
}

/* orc_step with the update fed bf16(g_bar) when gbar_bf16 is non-zero. */
int orc_step_fmt(orc_segment *segs, int32_t n_segs, int32_t R, const orc_hparams *hp,
                 int gbar_bf16, double *norm_out)
{
    if (R < 1 || n_segs < 0 || hp->step < 1)
        return ORC_INVALID;
    double norm = orc_grad_norm(segs, n_segs, R);
    if (norm_out)
        *norm_out = norm;
    if (!isfinite(norm))
        return ORC_NONFINITE;
    double c = orc_clip_coef(norm, hp->max_grad_norm);
    double bc1, bc2;
    bias_corrections(hp, &bc1, &bc2);
    for (int32_t s = 0; s < n_segs; ++s) {
        orc_segment *sg = &segs[s];
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < sg->numel; ++i)
            update_one(&sg->master[i], &sg->exp_avg[i], &sg->exp_avg_sq[i],
                       &sg->param_bf16[i],
                       update_gradient(orc_mean_grad(sg->grads, R, i), gbar_bf16),
                       c, hp, bc1, bc2);
    }
    return ORC_OK;
}

/* Steps 1, 4 and 5 at n independent points whose clip coefficient is already
 * known (for sampled checks of large states).  g_rows holds the R BF16
 * gradients of point k at g_rows[k * R + r]. */
void orc_update_points(int64_t n, const float *p, const float *m, const float *v,
                       const uint16_t *g_rows, int32_t R, double clip_coef,
                       const orc_hparams *hp, float *p_out, float *m_out,
                       float *v_out, uint16_t *pb_out)
{
    orc_update_points_fmt(n, p, m, v, g_rows, R, clip_coef, hp, 0,
                          p_out, m_out, v_out, pb_out);
}

/* orc_update_points with the update fed bf16(g_bar) when gbar_bf16 is set. */
void orc_update_points_fmt(int64_t n, const float *p, const float *m, const float *v,
                           const uint16_t *g_rows, int32_t R, double clip_coef,
                           const orc_hparams *hp, int gbar_bf16, float *p_out,
                           float *m_out, float *v_out, uint16_t *pb_out)
{
    double bc1, bc2;
    bias_corrections(hp, &bc1, &bc2);
    if (R < 1 || R > ORC_MAX_RANKS)
        return;
    for (int64_t k = 0; k < n; ++k) {
        const uint16_t *rows[ORC_MAX_RANKS];
        for (int32_t r = 0; r < R; ++r)
            rows[r] = &g_rows[k * R + r];
        float g_bar = update_gradient(orc_mean_grad(rows, R, 0), gbar_bf16);
        p_out[k] = p[k];
        m_out[k] = m[k];
        v_out[k] = v[k];
        update_one(&p_out[k], &m_out[k], &v_out[k], &pb_out[k], g_bar,
                   clip_coef, hp, bc1, bc2);
    }
}

/* Steps 1, 4 and 5 over n consecutive elements whose clip coefficient is
 * already known, in place (for a full check of a state too large to step in
 * one call: the norm comes from orc_grad_norm over all of it).  grads holds
 * R pointers, each to the n BF16 gradients of one rank. */
void orc_update_given_clip(int64_t n, float *p, float *m, float *v, uint16_t *pb,
                           const uint16_t *const *grads, int32_t R, double clip_coef,
                           const orc_hparams *hp, int gbar_bf16)
{
    if (R < 1 || R > ORC_MAX_RANKS)
        return;
    double bc1, bc2;
    bias_corrections(hp, &bc1, &bc2);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        update_one(&p[i], &m[i], &v[i], &pb[i],
                   update_gradient(orc_mean_grad(grads, R, i), gbar_bf16), clip_coef, hp, bc1, bc2);
}

/* Threads of the OpenMP loops from now on (n >= 1); for timing only. */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
