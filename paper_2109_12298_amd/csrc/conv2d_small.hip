// Per-sample Conv2d gradients for samples small enough to sit whole in LDS
// (the MNIST network's convolutions, for example): one workgroup per sample.
//
// gW_n[co][ci][u][v] = s * sum_{oh,ow} GY_n[co][oh][ow] * X_n[ci][oh*sh+u-ph][ow*sw+v-pw]
// gb_n[co]           = s * sum_{oh,ow} GY_n[co][oh][ow]
// (the weight gradient of the cross-correlation restricted to sample n; the
// unfold's column order (ci, u, v) is the weight's own layout).
//
// The workgroup stages the sample's padded input planes (zero halo) and its
// backprop [co][position] in LDS with every global load in flight at once,
// plus a table of each output position's offset in the padded plane.  The
// contraction over positions then runs on v_mfma_f32_16x16x4_f32 in 16 (kk)
// x 16 (co) blocks, each wave holding up to eight blocks' accumulators: a
// lane's operand is one LDS read of the unfold (its kk's plane offset + the
// position's offset) and one of the backprop; the unfold is never formed.  A lane's four
// accumulators are four consecutive kk of one co, stored as one float4.  The
// bias sums and the sample's squared norm are added in a fixed order, so the
// norm goes straight to sqnorm[n] (no partials).  Against the general kernel
// this keeps a sample's fixed costs (one load round trip, no K split, no
// second pass) small, which is what bounds these tiny convolutions.  The
// body lives in conv2d_small_dev.hpp, shared with the grouped
// per-sample-gradient kernel.
#include "common.hpp"
#include "conv2d_small.hpp"
#include "conv2d_small_dev.hpp"

namespace dpg {
namespace {

using namespace csmall;

template <typename T, int BPW>
__global__ __launch_bounds__(kThreads) void conv_small_kernel(const T *__restrict__ X, const T *__restrict__ GY,
                                                              SmallShape s, float scale, float *__restrict__ gW,
                                                              float *__restrict__ gb, float *__restrict__ sqnorm)
{
    extern __shared__ __attribute__((aligned(16))) float lds[];
    conv_small_sample<T, BPW>(X, GY, s, scale, gW, gb, sqnorm, blockIdx.x, lds);
}

template <int BPW>
void launch_small(const ConvSmallArgs &a, const SmallShape &s, bool bf16, float scale, float *gW, float *gb,
                  float *sqnorm, size_t lds, hipStream_t stream)
{
    if (bf16)
        conv_small_kernel<uint16_t, BPW><<<(unsigned)a.N, kThreads, lds, stream>>>(
            (const uint16_t *)a.X, (const uint16_t *)a.GY, s, scale, gW, gb, sqnorm);
    else
        conv_small_kernel<float, BPW><<<(unsigned)a.N, kThreads, lds, stream>>>(
            (const float *)a.X, (const float *)a.GY, s, scale, gW, gb, sqnorm);
}

}  // namespace

bool conv_small_ok(const ConvSmallArgs &a)
{
    SmallShape s;
    return make_small(a, s);
}

void conv_small_launch(const ConvSmallArgs &a, bool bf16, float scale, float *gW, float *gb, float *sqnorm,
                       hipStream_t stream)
{
    SmallShape s;
    make_small(a, s);
    s.vec = s.KK % 4 == 0 && aligned(gW, 16);
    s.xdma = s.xplain && !bf16 && aligned(a.X, 16);
    s.gdma = s.gplain && !bf16 && aligned(a.GY, 16);
    const size_t lds = (size_t)lds_floats(s) * sizeof(float);
    switch (s.bpw) {
    case 1: launch_small<1>(a, s, bf16, scale, gW, gb, sqnorm, lds, stream); break;
    case 2: launch_small<2>(a, s, bf16, scale, gW, gb, sqnorm, lds, stream); break;
    case 4: launch_small<4>(a, s, bf16, scale, gW, gb, sqnorm, lds, stream); break;
    default: launch_small<8>(a, s, bf16, scale, gW, gb, sqnorm, lds, stream); break;
    }
}

}  // namespace dpg
