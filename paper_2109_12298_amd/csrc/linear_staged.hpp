// Staged fp32 per-sample gradients of Linear layers over a sequence
// (linear.hip): the grouped launch that dp_grad_sample_many uses.
#pragma once

#include "common.hpp"

namespace dpg {

// The shapes dp_grad_sample_linear runs on its staged fp32 kernel (T a
// multiple of 16, d_in and d_out multiples of 4, 16-byte aligned A, B, gW),
// small enough that 16 of them fit one launch's grid.
bool fp32_staged_ok(const void *A, const void *B, const void *gW, i64 N, i64 T, i64 din, i64 dout);
// squared-norm partials per sample (one per 64 x 64 tile)
int fp32_staged_parts(i64 din, i64 dout);

// Several such layers sharing N, in one launch plus one launch adding each
// layer's squared-norm partials into its sqnorm row.  partial: N *
// fp32_staged_parts(din, dout) floats of scratch per layer (unused when
// sqnorm is NULL).
constexpr int kPsGroupMax = 16;
struct Fp32GroupLayer {
    const void *A, *B;
    i64 T, din, dout;
    float scale;
    float *gW, *gb, *sqnorm, *partial;
};
void fp32_grad_sample_group(const Fp32GroupLayer *layers, int count, i64 N, hipStream_t stream);

}  // namespace dpg
