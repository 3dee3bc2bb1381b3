/*
 * CPU oracle for the aggregate -> global-norm clip -> AdamW -> BF16 re-emit
 * update.  TEST INFRASTRUCTURE ONLY: it is called by the test suite, by the
 * smoke check and by the benchmark's CPU-baseline leg, never by the library.
 * It shares no code, header, table or constant with the HIP path.
 *
 * Everything is evaluated in FP64 from the stored FP32 / BF16 inputs and each
 * output is rounded once.  Parity pins (closed forms, invariants, library
 * cross-checks, brute force) live in the tests next to it.
 */
#ifndef SDP_ORACLE_H
#define SDP_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One flat layer state (Background, training-state table: BF16 weights and
 * gradients, FP32 master and two FP32 moments). */
typedef struct {
    float *master;
    float *exp_avg;
    float *exp_avg_sq;
    uint16_t *param_bf16;
    const uint16_t *const *grads; /* R pointers, one per data-parallel rank */
    int64_t numel;
} orc_segment;

typedef struct {
    double lr, beta1, beta2, eps, weight_decay, max_grad_norm;
    int64_t step; /* t >= 1 */
} orc_hparams;

enum { ORC_OK = 0, ORC_NONFINITE = 1, ORC_INVALID = -1 };
enum { ORC_MAX_RANKS = 64 };

uint16_t orc_bf16_from_f32(float x);
float orc_f32_from_bf16(uint16_t b);
void orc_bf16_array(const float *x, uint16_t *out, int64_t n);

float orc_mean_grad(const uint16_t *const *grads, int32_t R, int64_t i);
void orc_mean_grads(const uint16_t *const *grads, int32_t R, int64_t n, float *out);

double orc_grad_norm(const orc_segment *segs, int32_t n_segs, int32_t R);
double orc_sum_squares_f32(const float *x, int64_t n);
double orc_clip_coef(double norm, double max_grad_norm);

void orc_adamw_f64(int64_t n, const double *p, const double *m, const double *v,
                   const double *g, const orc_hparams *hp,
                   double *p_out, double *m_out, double *v_out);

int orc_step(orc_segment *segs, int32_t n_segs, int32_t R, const orc_hparams *hp,
             double *norm_out);
/* gbar_bf16 != 0: the update consumes bf16(g_bar); the norm still uses g_bar. */
int orc_step_fmt(orc_segment *segs, int32_t n_segs, int32_t R, const orc_hparams *hp,
                 int gbar_bf16, double *norm_out);

void orc_update_points(int64_t n, const float *p, const float *m, const float *v,
                       const uint16_t *g_rows, int32_t R, double clip_coef,
                       const orc_hparams *hp, float *p_out, float *m_out,
                       float *v_out, uint16_t *pb_out);
void orc_update_points_fmt(int64_t n, const float *p, const float *m, const float *v,
                           const uint16_t *g_rows, int32_t R, double clip_coef,
                           const orc_hparams *hp, int gbar_bf16, float *p_out,
                           float *m_out, float *v_out, uint16_t *pb_out);

void orc_update_given_clip(int64_t n, float *p, float *m, float *v, uint16_t *pb,
                           const uint16_t *const *grads, int32_t R, double clip_coef,
                           const orc_hparams *hp, int gbar_bf16);

int orc_num_threads(void);
void orc_set_num_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
