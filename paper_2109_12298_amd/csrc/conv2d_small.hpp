// One-workgroup-per-sample Conv2d per-sample gradients (conv2d_small.hip).
#pragma once

#include "common.hpp"

namespace dpg {

struct ConvSmallArgs {
    const void *X, *GY;
    i64 N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
};

// the kernel choice of dp_conv2d_set_path in force
int conv_path();

// the sample's padded planes, backprop and position table fit the LDS budget
bool conv_small_ok(const ConvSmallArgs &a);
// writes gW, gb (if not null) and sqnorm[n] (if not null) directly
void conv_small_launch(const ConvSmallArgs &a, bool bf16, float scale, float *gW, float *gb, float *sqnorm,
                       hipStream_t stream);

}  // namespace dpg
