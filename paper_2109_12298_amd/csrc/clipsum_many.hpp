// Grouped bf16 fused clipped sum (clipsum_many.hip).
#pragma once

#include "common.hpp"

namespace dpg {

constexpr int kClipManyMax = 16;   // layers per grouped launch

struct ClipManyItem {
    const void *A;
    const void *B;
    float *W;
    float *b;
    i64 din, dout, T;
    float scale;
};

// The grouped kernel takes bf16 layers with T a multiple of 32, N*T/32 < 2^31,
// d_in and d_out multiples of 8 and 16-byte aligned operands and sums.
bool clip_many_item_ok(const void *A, const void *B, const float *W, const float *bsum, i64 N, i64 T, i64 din,
                       i64 dout);
void clip_many_launch(const ClipManyItem *items, int count, i64 N, const float *norm, float C, hipStream_t stream);

}  // namespace dpg
