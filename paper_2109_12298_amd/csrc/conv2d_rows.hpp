// Row-chunked Conv2d per-sample gradients (conv2d_rows.hip), for samples
// whose input planes do not fit one workgroup's LDS.
#pragma once

#include "common.hpp"

namespace dpg {

struct ConvRowsArgs {
    const void *X, *GY;
    i64 N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
};

// a chunk of at least one output row fits the LDS budget
bool conv_rows_ok(const ConvRowsArgs &a);
// ... and the automatic choice prefers it to the tiled kernel: tiles of at
// least four 32-column blocks (with fewer, most of the four waves' position
// work feeds no MFMA; measured on the CIFAR network's first layer)
bool conv_rows_preferred(const ConvRowsArgs &a);
// gradient tiles per sample (norm partials in the workspace when above one)
int conv_rows_tiles(const ConvRowsArgs &a);
// writes gW, gb (if not null) and sqnorm (if not null; partial: N * tiles
// floats of workspace when there are several tiles)
void conv_rows_launch(const ConvRowsArgs &a, bool bf16, float scale, float *gW, float *gb, float *sqnorm,
                      float *partial, hipStream_t stream);

}  // namespace dpg
