// Staged bf16 per-sample gradients of a Linear layer (grad_sample_bf16.hip).
#pragma once

#include "common.hpp"

namespace dpg {

// T a multiple of 32, d_in and d_out multiples of 8, 16-byte aligned A, B, gW.
bool bf16_staged_ok(const void *A, const void *B, const void *gW, i64 N, i64 T, i64 din, i64 dout);
// squared-norm partials per sample (the caller adds them with sum_partials)
int bf16_staged_parts(i64 din, i64 dout);
void bf16_grad_sample_staged(const void *A, const void *B, i64 N, i64 T, i64 din, i64 dout, float scale, float *gW,
                             float *gb, float *partial, hipStream_t stream);

// Several such layers (each bf16_staged_ok) sharing N, in one launch plus
// one launch adding each layer's squared-norm partials into its sqnorm row.
// partial: N * bf16_staged_parts(din, dout) floats of scratch per layer
// (unused when sqnorm is NULL).
constexpr int kBf16GroupMax = 16;
struct Bf16GroupLayer {
    const void *A, *B;
    i64 T, din, dout;
    float scale;
    float *gW, *gb, *sqnorm, *partial;
};
void bf16_grad_sample_group(const Bf16GroupLayer *layers, int count, i64 N, hipStream_t stream);

}  // namespace dpg
