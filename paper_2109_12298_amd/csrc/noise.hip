// Gaussian noise and averaging: out = (sum + sigma * C * z) / denom.
//
// z is a counter-based stream: Philox4x32-10 (Salmon, Moraes, Dror, Shaw,
// "Parallel Random Numbers: As Easy as 1, 2, 3", SC'11) keyed by the 64-bit
// seed, with counter (e/4, param_index, step_lo, step_hi) for element e, so
// every element's noise is a pure function of (seed, step, param_index, e):
// no generator state, free resumption, and every data-parallel rank would
// draw identical noise without communicating.  Each 4-word block gives four
// normals by the Box-Muller transform on word pairs (w0, w1) and (w2, w3).
#include "common.hpp"
#include "philox.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void add_noise_kernel(const float *__restrict__ sum,
                                                             float *__restrict__ out, i64 numel,
                                                             uint32_t k0, uint32_t k1,
                                                             uint32_t pidx, uint32_t s_lo,
                                                             uint32_t s_hi, float sc, float denom,
                                                             bool noise, bool vec)
{
    const i64 q = (i64)blockIdx.x * kThreads + threadIdx.x;
    const i64 e0 = 4 * q;
    if (e0 >= numel) return;
    float z[4] = {0.f, 0.f, 0.f, 0.f};
    uint32_t w[4];
    if (noise) normals4(q, pidx, s_lo, s_hi, k0, k1, z, w);
    if (vec && e0 + 4 <= numel) {
        const float4 s = reinterpret_cast<const float4 *>(sum)[q];
        float4 o;
        o.x = (s.x + sc * z[0]) / denom;
        o.y = (s.y + sc * z[1]) / denom;
        o.z = (s.z + sc * z[2]) / denom;
        o.w = (s.w + sc * z[3]) / denom;
        reinterpret_cast<float4 *>(out)[q] = o;
    } else {
        for (int i = 0; i < 4 && e0 + i < numel; ++i) out[e0 + i] = (sum[e0 + i] + sc * z[i]) / denom;
    }
}

__global__ __launch_bounds__(kThreads) void normals_kernel(float *__restrict__ z,
                                                           uint32_t *__restrict__ raw, i64 numel,
                                                           uint32_t k0, uint32_t k1, uint32_t pidx,
                                                           uint32_t s_lo, uint32_t s_hi)
{
    const i64 q = (i64)blockIdx.x * kThreads + threadIdx.x;
    const i64 e0 = 4 * q;
    if (e0 >= numel) return;
    float zz[4];
    uint32_t w[4];
    normals4(q, pidx, s_lo, s_hi, k0, k1, zz, w);
    for (int i = 0; i < 4 && e0 + i < numel; ++i) {
        if (z) z[e0 + i] = zz[i];
        if (raw) raw[e0 + i] = w[i];
    }
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" dp_status dp_add_noise(const float *sum, float *out, int64_t numel, uint64_t seed,
                                  uint64_t step, uint32_t param_index, float sigma, float C,
                                  float denom, int32_t *status, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(numel >= 0, DP_EINVAL);
    DPG_REQUIRE(numel == 0 || (sum != nullptr && out != nullptr), DP_EINVAL);
    DPG_REQUIRE(sigma >= 0.0f && denom > 0.0f && C > 0.0f, DP_EINVAL);
    DPG_REQUIRE(!(sigma > 0.0f && __builtin_isinf(C)), DP_EINVAL);
    DPG_REQUIRE(numel / 4 < (i64(1) << 32), DP_EINVAL);   // block index must fit the counter word
    if (numel == 0) return DP_OK;
    const bool noise = sigma > 0.0f;
    const bool vec = ((reinterpret_cast<uintptr_t>(sum) | reinterpret_cast<uintptr_t>(out)) & 15) == 0;
    const i64 nq = ceil_div(numel, 4);
    add_noise_kernel<<<(unsigned)ceil_div(nq, kThreads), kThreads, 0, stream>>>(
        sum, out, numel, (uint32_t)seed, (uint32_t)(seed >> 32), param_index, (uint32_t)step,
        (uint32_t)(step >> 32), noise ? sigma * C : 0.0f, denom, noise, vec);
    return launch_status();
}

extern "C" dp_status dp_philox_normals(float *z, uint32_t *raw, int64_t numel, uint64_t seed,
                                       uint64_t step, uint32_t param_index, hipStream_t stream)
{
    DPG_REQUIRE(numel >= 0, DP_EINVAL);
    DPG_REQUIRE(numel / 4 < (i64(1) << 32), DP_EINVAL);
    if (numel == 0 || (z == nullptr && raw == nullptr)) return DP_OK;
    const i64 nq = ceil_div(numel, 4);
    normals_kernel<<<(unsigned)ceil_div(nq, kThreads), kThreads, 0, stream>>>(
        z, raw, numel, (uint32_t)seed, (uint32_t)(seed >> 32), param_index, (uint32_t)step,
        (uint32_t)(step >> 32));
    return launch_status();
}
