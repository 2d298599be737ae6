// GroupNorm / InstanceNorm affine per-sample gradients.  Both normalize
// [N][C][spatial] inputs within each sample (over a group of channels, or
// over one channel) and then apply a per-channel affine y = gamma[c] * xhat
// + beta[c]; neither mixes samples, so their per-sample gradients exist
// (unlike BatchNorm's).  With the normalized input xhat given:
//   ggamma_n[c] = s * sum_p B[n][c][p] * xhat[n][c][p]
//   gbeta_n[c]  = s * sum_p B[n][c][p]
// over the channel's P spatial positions, which are contiguous in memory.
// A wave reduces one channel at a time (lanes over the positions, 16-byte
// loads when the rows allow, then a fixed tree), or, for planes of at most 64
// positions, four channels at a time on 16 lanes each; the sums are
// deterministic.  A workgroup takes 16 channels of one sample, and the
// sample's squared norm is added over its channel blocks in block order.
#include "common.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kChanPerBlock = 16;

template <typename T>
__device__ __forceinline__ float4 ld4(const T *p);

template <>
__device__ __forceinline__ float4 ld4<float>(const float *p)
{
    return *reinterpret_cast<const float4 *>(p);
}

template <>
__device__ __forceinline__ float4 ld4<uint16_t>(const uint16_t *p)
{
    const uint2 u = *reinterpret_cast<const uint2 *>(p);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

// sum over the LPC lanes of a segment (a fixed butterfly; every lane of the
// segment ends with the sum)
template <int LPC>
__device__ __forceinline__ float seg_sum(float v)
{
    if constexpr (LPC == 64) return wave_sum(v);
#pragma unroll
    for (int o = LPC / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// VEC: P % 4 == 0 and 16-byte (fp32) / 8-byte (bf16) aligned rows.
// LPC: lanes per channel (64, or 16 for planes of at most 64 positions)
template <typename T, bool VEC, int LPC>
__global__ __launch_bounds__(kThreads) void gn_affine_kernel(const T *__restrict__ xh, const T *__restrict__ B,
                                                             i64 C, i64 P, int cblocks, float scale,
                                                             float *__restrict__ gg, float *__restrict__ gbt,
                                                             float *__restrict__ sqout, int direct)
{
    __shared__ float red[kWaves];
    const i64 n = blockIdx.x / cblocks;
    const int cb = (int)(blockIdx.x % cblocks);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    constexpr int SEGS = 64 / LPC;                 // channels a wave takes at once
    const int seg = lane / LPC, sl = lane % LPC;
    float sq = 0.0f;
    for (int k = wave * SEGS; k < kChanPerBlock; k += kWaves * SEGS) {
        const i64 c = (i64)cb * kChanPerBlock + k + seg;
        const bool live = c < C;
        const T *x = xh + (n * C + (live ? c : 0)) * P;
        const T *b = B + (n * C + (live ? c : 0)) * P;
        float ag = 0.0f, ab = 0.0f;
        if (live) {
            if (VEC) {
                for (i64 p = 4 * sl; p < P; p += 4 * LPC) {
                    const float4 bv = ld4<T>(b + p), xv = ld4<T>(x + p);
                    ag += bv.x * xv.x + bv.y * xv.y + bv.z * xv.z + bv.w * xv.w;
                    ab += bv.x + bv.y + bv.z + bv.w;
                }
            } else {
                for (i64 p = sl; p < P; p += LPC) {
                    const float bv = load_elem<T>(b, p);
                    ag += bv * load_elem<T>(x, p);
                    ab += bv;
                }
            }
        }
        ag = seg_sum<LPC>(ag);
        ab = seg_sum<LPC>(ab);
        if (live && sl == 0) {
            const float g = scale * ag, e = scale * ab;
            gg[n * C + c] = g;
            if (gbt) gbt[n * C + c] = e;
            sq += g * g + (gbt ? e * e : 0.0f);
        }
    }
    sq = wave_sum(sq);                             // the segments' shares (one lane each), in a fixed order
    if (lane == 0) red[wave] = sq;
    __syncthreads();
    if (threadIdx.x == 0 && sqout) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += red[w];
        if (direct) sqout[n] = t;
        else sqout[n * cblocks + cb] = t;
    }
}

template <typename T>
void launch_gn(bool vec, bool narrow, dim3 grid, const void *xh, const void *B, i64 C, i64 P, int cblocks,
               float scale, float *gg, float *gbt, float *sqout, int direct, hipStream_t stream)
{
    const T *x = (const T *)xh, *b = (const T *)B;
    if (vec && narrow)
        gn_affine_kernel<T, true, 16><<<grid, kThreads, 0, stream>>>(x, b, C, P, cblocks, scale, gg, gbt, sqout, direct);
    else if (vec)
        gn_affine_kernel<T, true, 64><<<grid, kThreads, 0, stream>>>(x, b, C, P, cblocks, scale, gg, gbt, sqout, direct);
    else if (narrow)
        gn_affine_kernel<T, false, 16><<<grid, kThreads, 0, stream>>>(x, b, C, P, cblocks, scale, gg, gbt, sqout,
                                                                      direct);
    else
        gn_affine_kernel<T, false, 64><<<grid, kThreads, 0, stream>>>(x, b, C, P, cblocks, scale, gg, gbt, sqout,
                                                                      direct);
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_grad_sample_groupnorm_workspace_bytes(int64_t N, int64_t C, int64_t P)
{
    if (N <= 0 || C <= 0 || P < 0) return 0;
    const i64 cblocks = ceil_div(C, (i64)kChanPerBlock);
    return cblocks > 1 ? (size_t)(N * cblocks) * sizeof(float) : 0;
}

extern "C" dp_status dp_grad_sample_groupnorm(const void *xhat, const void *B, dp_dtype dt, int64_t N, int64_t C,
                                              int64_t P, float scale, float *ggamma, float *gbeta, float *sqnorm,
                                              int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && C >= 1 && P >= 0, DP_EINVAL);
    DPG_REQUIRE(N * C < (i64(1) << 40) && C * P < (i64(1) << 40), DP_EINVAL);
    DPG_REQUIRE(N == 0 || ggamma != nullptr, DP_EINVAL);
    DPG_REQUIRE(N == 0 || P == 0 || (xhat != nullptr && B != nullptr), DP_EINVAL);
    const size_t need = dp_grad_sample_groupnorm_workspace_bytes(N, C, P);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;
    const int cblocks = (int)ceil_div(C, (i64)kChanPerBlock);
    const int direct = cblocks == 1;
    float *sqout = sqnorm ? (direct ? sqnorm : (float *)ws) : nullptr;
    const dim3 grid((unsigned)(N * cblocks));
    const bool bf = dt == DP_BF16;
    const bool vec = P % 4 == 0 && aligned(xhat, bf ? 8 : 16) && aligned(B, bf ? 8 : 16);
    const bool narrow = P <= 64;                   // four channels per wave, 16 lanes each
    if (bf) launch_gn<uint16_t>(vec, narrow, grid, xhat, B, C, P, cblocks, scale, ggamma, gbeta, sqout, direct,
                                stream);
    else launch_gn<float>(vec, narrow, grid, xhat, B, C, P, cblocks, scale, ggamma, gbeta, sqout, direct, stream);
    if (sqnorm && !direct) sum_partials((const float *)ws, N, cblocks, sqnorm, stream);
    return launch_status();
}
