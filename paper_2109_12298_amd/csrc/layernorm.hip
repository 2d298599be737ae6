// LayerNorm affine per-sample gradients: for y = gamma * xhat + beta,
//   ggamma_n[k] = s * sum_t B[n][t][k] * xhat[n][t][k],  gbeta_n[k] = s * sum_t B[n][t][k].
// Column sums over positions, HBM-bound.  Positions are split into ranges so
// that small batches still fill the GPU; a second pass adds the range
// partials in range order and forms each sample's squared norm.
#include "common.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;

template <typename T>
__global__ __launch_bounds__(kThreads) void ln_partial_kernel(const T *__restrict__ xh,
                                                              const T *__restrict__ B, i64 Tn,
                                                              i64 D, int splits, i64 per,
                                                              float *__restrict__ part)
{
    const i64 n = blockIdx.x / splits;
    const int sp = blockIdx.x % splits;
    const i64 t0 = (i64)sp * per;
    const i64 t1 = t0 + per < Tn ? t0 + per : Tn;
    float *pg = part + ((i64)n * splits + sp) * 2 * D;
    for (i64 k = threadIdx.x; k < D; k += kThreads) {
        float ag = 0.0f, ab = 0.0f;
        for (i64 t = t0; t < t1; ++t) {
            const i64 idx = (n * Tn + t) * D + k;
            const float b = load_elem<T>(B, idx);
            ag += b * load_elem<T>(xh, idx);
            ab += b;
        }
        pg[k] = ag;
        pg[D + k] = ab;
    }
}

__global__ __launch_bounds__(kThreads) void ln_finish_kernel(const float *__restrict__ part,
                                                             i64 D, int splits, float scale,
                                                             float *__restrict__ gg,
                                                             float *__restrict__ gbt,
                                                             float *__restrict__ sqnorm)
{
    __shared__ float red[16];
    const i64 n = blockIdx.x;
    float sq = 0.0f;
    for (i64 k = threadIdx.x; k < D; k += kThreads) {
        float ag = 0.0f, ab = 0.0f;
        for (int sp = 0; sp < splits; ++sp) {
            const float *pg = part + ((i64)n * splits + sp) * 2 * D;
            ag += pg[k];
            ab += pg[D + k];
        }
        ag *= scale;
        ab *= scale;
        gg[n * D + k] = ag;
        gbt[n * D + k] = ab;
        sq += ag * ag + ab * ab;
    }
    sq = block_sum(sq, red);
    if (sqnorm && threadIdx.x == 0) sqnorm[n] = sq;
}

void ln_split(i64 T, int *splits, i64 *per)
{
    i64 s = ceil_div(T, 16);
    if (s > 64) s = 64;
    if (s < 1) s = 1;
    *per = T > 0 ? ceil_div(T, s) : 1;
    *splits = T > 0 ? (int)ceil_div(T, *per) : 1;
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_grad_sample_layernorm_workspace_bytes(int64_t N, int64_t T, int64_t D)
{
    if (N <= 0 || T < 0 || D <= 0) return 0;
    int splits;
    i64 per;
    ln_split(T, &splits, &per);
    return (size_t)(N * splits * 2 * D) * sizeof(float);
}

extern "C" dp_status dp_grad_sample_layernorm(const void *xhat, const void *B, dp_dtype dt,
                                              int64_t N, int64_t T, int64_t D, float scale,
                                              float *ggamma, float *gbeta, float *sqnorm,
                                              int32_t *status, void *ws, size_t ws_bytes,
                                              hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && T >= 0 && D >= 1, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (ggamma != nullptr && gbeta != nullptr), DP_EINVAL);
    DPG_REQUIRE(N * T == 0 || (xhat != nullptr && B != nullptr), DP_EINVAL);
    const size_t need = dp_grad_sample_layernorm_workspace_bytes(N, T, D);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;
    int splits;
    i64 per;
    ln_split(T, &splits, &per);
    float *part = (float *)ws;
    if (T > 0) {
        const dim3 grid((unsigned)(N * splits));
        if (dt == DP_F32)
            ln_partial_kernel<float><<<grid, kThreads, 0, stream>>>((const float *)xhat, (const float *)B,
                                                                    T, D, splits, per, part);
        else
            ln_partial_kernel<uint16_t><<<grid, kThreads, 0, stream>>>(
                (const uint16_t *)xhat, (const uint16_t *)B, T, D, splits, per, part);
    } else {
        zero_fill(part, N * splits * 2 * D, stream);
    }
    ln_finish_kernel<<<(unsigned)N, kThreads, 0, stream>>>(part, D, splits, scale, ggamma, gbeta, sqnorm);
    return launch_status();
}
