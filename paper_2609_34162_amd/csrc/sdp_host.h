// Host lanes of libsdp that run on CPU cores: the AdamW update of the
// host-update route.  Plain C++ (no HIP types), compiled on its own with the
// host compiler and -ffp-contract=off.  Not installed; not part of the ABI.
#pragma once

#include <stdint.h>

namespace sdp_host {

// Per-step constants of the update, computed once in FP64 (the same values
// the fused GPU update receives), plus the clip coefficient c.
struct AdamConsts {
    double c;
    double lr_wd;  // lr * weight_decay
    double beta1, one_minus_beta1;
    double beta2, one_minus_beta2;
    double step_size;  // lr / (1 - beta1^t)
    double inv_bc2;    // 1 / (1 - beta2^t)
    double eps;
};

// One flat run of host state and the mean gradient that feeds it: FP32
// (gbar_bf16 == 0) or BF16 bit patterns (gbar_bf16 != 0).
struct AdamArgs {
    float *p, *m, *v;
    uint16_t *pb;
    const void *gbar;
    int gbar_bf16;
};

// Instruction sets of adamw_range.
enum Simd { kScalar = 0, kAvx512 = 1 };

// The best instruction set this CPU runs (kAvx512 needs AVX-512 F/BW/VL/DQ).
int simd_best();

// dst[i] = BF16 round-to-nearest-even of src[i] for n values: NaN keeps sign
// and top payload bits and gets the quiet bit, infinities are kept, overflow
// of the largest values rounds to infinity.  AVX-512 where simd_best() has it.
void cast_bf16(const float *src, uint16_t *dst, int64_t n);

// Updates elements [i0, i1) of a in place.  simd above simd_best() is
// lowered to it.  Results do not depend on simd, i0 or i1: each element is
// computed on its own with the same sequence of IEEE operations, under the
// default rounding mode with denormals kept (set for the call and restored).
void adamw_range(const AdamArgs &a, const AdamConsts &k, int64_t i0, int64_t i1, int simd);

}  // namespace sdp_host
