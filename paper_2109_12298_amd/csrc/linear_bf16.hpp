// bf16 MFMA path of the Linear entry points (linear_bf16.hip).
#pragma once

#include "common.hpp"

namespace dpg {

// The bf16 kernels need T > 1, d_in and d_out multiples of 8 and 16-byte aligned pointers.
bool bf16_path_ok(const void *A, const void *B, const void *out, i64 T, i64 din, i64 dout);
int bf16_tiles(i64 din, i64 dout);
void bf16_grad_sample(const void *A, const void *B, i64 N, i64 T, i64 din, i64 dout, float scale, float *gW,
                      float *gb, float *partial, hipStream_t stream);
size_t bf16_clip_workspace(i64 N, i64 T, i64 din, i64 dout);
void bf16_clip_accumulate(const void *A, const void *B, i64 N, i64 T, i64 din, i64 dout, float scale,
                          const float *norm, float C, float *sumW, float *sumb, void *ws, hipStream_t stream);

}  // namespace dpg
