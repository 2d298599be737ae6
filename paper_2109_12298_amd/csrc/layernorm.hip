// LayerNorm affine per-sample gradients: for y = gamma * xhat + beta,
//   ggamma_n[k] = s * sum_t B[n][t][k] * xhat[n][t][k],  gbeta_n[k] = s * sum_t B[n][t][k].
// Column sums over positions, HBM-bound.  Positions are split into ranges so
// that small batches still fill the GPU; a second pass adds the range
// partials in range order and forms each sample's squared norm.
#include "common.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;

// four consecutive features of one row as fp32
template <typename T>
__device__ __forceinline__ float4 load4f(const T *p);

template <>
__device__ __forceinline__ float4 load4f<float>(const float *p)
{
    return *reinterpret_cast<const float4 *>(p);
}

template <>
__device__ __forceinline__ float4 load4f<uint16_t>(const uint16_t *p)
{
    const uint2 u = *reinterpret_cast<const uint2 *>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

// Vector path (D % 4 == 0, aligned rows): a thread owns four features and
// keeps four rows' loads in flight; rows are still added in ascending t.
template <typename T>
__global__ __launch_bounds__(kThreads) void ln_partial_vec_kernel(const T *__restrict__ xh,
                                                                  const T *__restrict__ B, i64 Tn,
                                                                  i64 D, int splits, i64 per,
                                                                  float *__restrict__ part)
{
    const i64 n = blockIdx.x / splits;
    const int sp = blockIdx.x % splits;
    const i64 t0 = (i64)sp * per;
    const i64 t1 = t0 + per < Tn ? t0 + per : Tn;
    float *pg = part + ((i64)n * splits + sp) * 2 * D;
    for (i64 k = 4 * (i64)threadIdx.x; k < D; k += 4 * kThreads) {
        float4 ag = make_float4(0.f, 0.f, 0.f, 0.f), ab = ag;
        i64 t = t0;
        for (; t + 4 <= t1; t += 4) {
            float4 b[4], x[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const i64 idx = (n * Tn + t + r) * D + k;
                b[r] = load4f<T>(B + idx);
                x[r] = load4f<T>(xh + idx);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                ag.x += b[r].x * x[r].x; ag.y += b[r].y * x[r].y; ag.z += b[r].z * x[r].z; ag.w += b[r].w * x[r].w;
                ab.x += b[r].x; ab.y += b[r].y; ab.z += b[r].z; ab.w += b[r].w;
            }
        }
        for (; t < t1; ++t) {
            const i64 idx = (n * Tn + t) * D + k;
            const float4 b = load4f<T>(B + idx), x = load4f<T>(xh + idx);
            ag.x += b.x * x.x; ag.y += b.y * x.y; ag.z += b.z * x.z; ag.w += b.w * x.w;
            ab.x += b.x; ab.y += b.y; ab.z += b.z; ab.w += b.w;
        }
        *reinterpret_cast<float4 *>(pg + k) = ag;
        *reinterpret_cast<float4 *>(pg + D + k) = ab;
    }
}

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
        const float *pg = part + (i64)n * splits * 2 * D;
        float ag = ordered_sum(pg + k, 2 * D, splits);
        float ab = ordered_sum(pg + D + k, 2 * D, splits);
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
        const bool vec = D % 4 == 0 && aligned(xhat, dt == DP_F32 ? 16 : 8) && aligned(B, dt == DP_F32 ? 16 : 8);
        if (vec && dt == DP_F32)
            ln_partial_vec_kernel<float><<<grid, kThreads, 0, stream>>>((const float *)xhat, (const float *)B,
                                                                        T, D, splits, per, part);
        else if (vec)
            ln_partial_vec_kernel<uint16_t><<<grid, kThreads, 0, stream>>>(
                (const uint16_t *)xhat, (const uint16_t *)B, T, D, splits, per, part);
        else if (dt == DP_F32)
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
