/* The C ABI used from plain C99: the header compiles on its own, and the
 * host-only entry points run without a GPU.  Prints the struct sizes and
 * offsets that the Python binding must agree with. */
#include <stddef.h>
#include <stdio.h>
#include <string.h>

#include "sdp.h"

#define FAILIF(c, msg)                                  \
    do {                                                \
        if (c) {                                        \
            fprintf(stderr, "FAIL: %s\n", msg);         \
            return 1;                                   \
        }                                               \
    } while (0)

int main(void) {
    /* layouts */
    printf("sdp_adamw_params %zu %zu\n", sizeof(sdp_adamw_params), offsetof(sdp_adamw_params, step));
    printf("sdp_segment %zu %zu %zu\n", sizeof(sdp_segment), offsetof(sdp_segment, n_ranks),
           offsetof(sdp_segment, numel));
    printf("sdp_kernel_times %zu %zu\n", sizeof(sdp_kernel_times), offsetof(sdp_kernel_times, host_adam_elems));
    printf("sdp_rates %zu %zu\n", sizeof(sdp_rates), offsetof(sdp_rates, dep_us));
    printf("sdp_prediction %zu %zu\n", sizeof(sdp_prediction), offsetof(sdp_prediction, n_chunks));

    /* host-only calls */
    int64_t numels[2] = {3 * SDP_NORM_TILE + 5, 1};
    int64_t chunks = 0, tiles = 0;
    FAILIF(sdp_plan(numels, 2, SDP_NORM_TILE, &chunks, &tiles) != SDP_OK, "sdp_plan");
    FAILIF(chunks != 5 || tiles != 5, "sdp_plan counts");
    FAILIF(strcmp(sdp_status_string(SDP_ERR_NONFINITE), "SDP_ERR_NONFINITE") != 0, "status string");
    FAILIF(sdp_plan(numels, 2, 1000, &chunks, &tiles) != SDP_ERR_INVALID_ARGUMENT, "bad chunk accepted");
    FAILIF(strlen(sdp_last_error()) == 0, "no error text");

    /* the host AdamW lane on 8 elements: zero gradient, lr = 0.5, wd = 0.1
     * -> p' = p (1 - 0.05) exactly for these values, moments stay 0 */
    static float p[8] = {2, -2, 4, 8, 0.5f, -0.5f, 1, 0};
    static float m[8], v[8], g[8];
    static uint16_t pb[8];
    sdp_adamw_params hp = {0.5, 0.9, 0.999, 1e-8, 0.1, 0.0, 1};
    FAILIF(sdp_host_adamw(NULL, p, m, v, pb, g, SDP_GBAR_F32, 8, 1.0, &hp) != SDP_OK, "sdp_host_adamw");
    FAILIF(p[0] != 1.9f || p[3] != 7.6f || p[7] != 0.0f || m[0] != 0.0f || v[0] != 0.0f, "host AdamW values");
    FAILIF(pb[0] != 0x3ff3, "BF16 of 1.9");

    /* the step-time model */
    sdp_rates r = {50, 40, 90, 0, 5000, 4000, 0, 0, 1e7, 0, 300, 0, 1, 0};
    sdp_prediction pr;
    FAILIF(sdp_predict_step(SDP_SCHED_STREAMED, numels, 2, 2, SDP_NORM_TILE, 0, &r, &pr) != SDP_OK, "predict");
    FAILIF(!(pr.predicted_ms >= pr.bound_ms && pr.n_chunks == 5), "prediction");
    printf("ok\n");
    return 0;
}
