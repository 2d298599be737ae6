// Grouped clipped sums and noise: every parameter tensor of a step in two
// launches instead of two per tensor.
//
// Pass 1 (column reduce, only for tensors given as per-sample gradients):
//   sum[e] = sum_n c_n * G[n][e] over contiguous sample ranges, n ascending;
//   one range writes the sum directly, several write range partials.
// Pass 2 (finish): adds the range partials in range order, stores the clipped
//   sum (summed_grad), and, when an output is given, writes
//   out[e] = (sum[e] + sigma * C * z[e]) / denom (grad) with z the tensor's
//   Philox stream.  The step may be read from device memory so that a
//   captured graph replays the call at an advancing step.
#include "common.hpp"
#include "philox.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxGroup = 40;

struct GroupDesc {
    int count;
    int splits;
    i64 per_split;
    i64 N;
    int cblocks;                   // total column-reduce workgroups per range
    int fblocks;                   // total finish workgroups
    const float *G[kMaxGroup];
    float *S[kMaxGroup];
    float *O[kMaxGroup];
    i64 numel[kMaxGroup];
    i64 ws_off[kMaxGroup];         // first partial of the tensor, in floats
    i64 stride[kMaxGroup];         // floats between two ranges' partials of the tensor
    int cblk0[kMaxGroup + 1];      // first column-reduce workgroup of each tensor
    int fblk0[kMaxGroup + 1];      // first finish workgroup of each tensor
    uint32_t pidx[kMaxGroup];
    uint32_t flags[kMaxGroup];     // bit 0: column-reduce vectorized, bit 1: finish vectorized
    uint8_t R[kMaxGroup];          // 1: the tensor's sum is formed here from per-sample grads
};

__device__ __forceinline__ int find_param(const int *blk0, int count, int b)
{
    int p = 0;
    while (p + 1 < count && blk0[p + 1] <= b) ++p;
    return p;
}

__global__ __launch_bounds__(kThreads) void colsum_many_kernel(GroupDesc d, const float *__restrict__ norm,
                                                               float C, float *__restrict__ ws)
{
    const int split = blockIdx.x / d.cblocks;
    const int b = blockIdx.x % d.cblocks;
    const int p = find_param(d.cblk0, d.count, b);
    const float *G = d.G[p];
    const i64 numel = d.numel[p];
    const int eb = b - d.cblk0[p];
    const i64 n0 = (i64)split * d.per_split;
    const i64 n1 = n0 + d.per_split < d.N ? n0 + d.per_split : d.N;
    float *o = d.splits > 1 ? ws + d.ws_off[p] + (i64)split * d.stride[p] : d.S[p];
    if (d.flags[p] & 1u) {
        const i64 e4 = (i64)eb * kThreads + threadIdx.x;
        if (4 * e4 >= numel) return;
        const float4 *g = reinterpret_cast<const float4 *>(G) + e4;
        const i64 st = numel / 4;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        i64 n = n0;
        // eight samples' loads in flight before the (in-order) accumulation
        for (; n + 8 <= n1; n += 8) {
            float4 a[8];
            float c[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) a[j] = g[(n + j) * st];
#pragma unroll
            for (int j = 0; j < 8; ++j) c[j] = clip_factor(norm[n + j], C);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                acc.x += c[j] * a[j].x; acc.y += c[j] * a[j].y;
                acc.z += c[j] * a[j].z; acc.w += c[j] * a[j].w;
            }
        }
        for (; n < n1; ++n) {
            const float4 a = g[n * st];
            const float cn = clip_factor(norm[n], C);
            acc.x += cn * a.x; acc.y += cn * a.y; acc.z += cn * a.z; acc.w += cn * a.w;
        }
        reinterpret_cast<float4 *>(o)[e4] = acc;
    } else {
        const i64 e = (i64)eb * kThreads + threadIdx.x;
        if (e >= numel) return;
        float acc = 0.0f;
        for (i64 n = n0; n < n1; ++n) acc += clip_factor(norm[n], C) * G[n * numel + e];
        o[e] = acc;
    }
}

__global__ __launch_bounds__(kThreads) void finish_many_kernel(GroupDesc d, const float *__restrict__ ws,
                                                               uint32_t k0, uint32_t k1, uint64_t step,
                                                               const uint64_t *__restrict__ step_dev,
                                                               float sc, float denom, int noise)
{
    const int b = blockIdx.x;
    const int p = find_param(d.fblk0, d.count, b);
    const i64 numel = d.numel[p];
    const i64 q = (i64)(b - d.fblk0[p]) * kThreads + threadIdx.x;
    const i64 e0 = 4 * q;
    if (e0 >= numel) return;
    const bool col = d.R[p] != 0;
    const bool from_parts = col && d.splits > 1;
    const int cnt = e0 + 4 <= numel ? 4 : (int)(numel - e0);
    float s[4] = {0.f, 0.f, 0.f, 0.f};
    if (col && d.N == 0) {
        // empty batch: the clipped sum is zero
    } else if (from_parts) {
        // range partials are 16-byte aligned (per-range stride is a multiple of 4)
        const float *part = ws + d.ws_off[p] + e0;
        const i64 st = d.stride[p];
        int k = 0;
        for (; k + 8 <= d.splits; k += 8) {
            float4 v[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const float4 *>(part + (i64)(k + j) * st);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                s[0] += v[j].x; s[1] += v[j].y; s[2] += v[j].z; s[3] += v[j].w;
            }
        }
        for (; k < d.splits; ++k) {
            const float4 v = *reinterpret_cast<const float4 *>(part + (i64)k * st);
            s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
        }
    } else {
        for (int i = 0; i < cnt; ++i) s[i] = d.S[p][e0 + i];
    }
    if (col && (from_parts || d.N == 0)) {
        for (int i = 0; i < cnt; ++i) d.S[p][e0 + i] = s[i];
    }
    float *O = d.O[p];
    if (O == nullptr) return;
    float z[4] = {0.f, 0.f, 0.f, 0.f};
    if (noise) {
        const uint64_t st = step + (step_dev ? *step_dev : 0ull);
        uint32_t w[4];
        normals4(q, d.pidx[p], (uint32_t)st, (uint32_t)(st >> 32), k0, k1, z, w);
    }
    if ((d.flags[p] & 2u) && cnt == 4) {
        float4 o;
        o.x = (s[0] + sc * z[0]) / denom;
        o.y = (s[1] + sc * z[1]) / denom;
        o.z = (s[2] + sc * z[2]) / denom;
        o.w = (s[3] + sc * z[3]) / denom;
        reinterpret_cast<float4 *>(O)[q] = o;
    } else {
        for (int i = 0; i < cnt; ++i) O[e0 + i] = (s[i] + sc * z[i]) / denom;
    }
}

__global__ void step_advance_kernel(uint64_t *p, uint64_t by)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) *p += by;
}

// Build the descriptor of params[first, first+count) and the workspace it needs.
size_t describe(const dp_param *params, int first, int count, i64 N, GroupDesc &d)
{
    d.count = count;
    d.N = N;
    i64 col_blocks = 0;
    for (int i = 0; i < count; ++i) {
        const dp_param &q = params[first + i];
        if ((q.flags & DP_PARAM_REDUCE) && N > 0) {
            const bool v = (q.numel & 3) == 0;
            col_blocks += ceil_div(q.numel, v ? 4 * kThreads : kThreads);
        }
    }
    i64 want = col_blocks > 0 ? ceil_div(2048, col_blocks) : 1;
    i64 maxs = N / 16;
    if (want > maxs) want = maxs;
    if (want > 64) want = 64;
    if (want < 1) want = 1;
    d.per_split = N > 0 ? ceil_div(N, want) : 1;
    d.splits = N > 0 ? (int)ceil_div(N, d.per_split) : 1;
    size_t ws_floats = 0;
    int cb = 0, fb = 0;
    for (int i = 0; i < count; ++i) {
        const dp_param &q = params[first + i];
        d.R[i] = (q.flags & DP_PARAM_REDUCE) ? 1 : 0;
        d.G[i] = q.grad_sample;
        d.S[i] = q.sum;
        d.O[i] = q.out;
        d.numel[i] = q.numel;
        d.pidx[i] = q.param_index;
        d.stride[i] = (q.numel + 3) & ~i64(3);
        d.ws_off[i] = (i64)ws_floats;
        d.cblk0[i] = cb;
        d.fblk0[i] = fb;
        uint32_t f = 0;
        const bool col = (q.flags & DP_PARAM_REDUCE) && N > 0;
        if (col) {
            const bool to_ws = d.splits > 1;
            bool v = (q.numel & 3) == 0 && aligned(q.grad_sample, 16) && (to_ws || aligned(q.sum, 16));
            if (v) f |= 1u;
            cb += (int)ceil_div(q.numel, v ? 4 * kThreads : kThreads);
            if (to_ws) ws_floats += (size_t)d.splits * d.stride[i];
        }
        if ((q.numel & 3) == 0 && aligned(q.out, 16)) f |= 2u;
        d.flags[i] = f;
        fb += (int)ceil_div(ceil_div(q.numel, 4), kThreads);
    }
    d.cblk0[count] = cb;
    d.fblk0[count] = fb;
    d.cblocks = cb;
    d.fblocks = fb;
    return ws_floats * sizeof(float);
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_clip_noise_many_workspace_bytes(const dp_param *params, int32_t count, int64_t N)
{
    if (params == nullptr || count <= 0 || N < 0) return 0;
    size_t need = 0;
    for (int first = 0; first < count; first += kMaxGroup) {
        const int c = count - first < kMaxGroup ? count - first : kMaxGroup;
        GroupDesc d;
        const size_t b = describe(params, first, c, N, d);
        if (b > need) need = b;
    }
    return need;
}

extern "C" dp_status dp_clip_noise_many(const dp_param *params, int32_t count, int64_t N, const float *norm,
                                        float C, uint64_t seed, uint64_t step, const uint64_t *step_dev,
                                        float sigma, float denom, int32_t *status, void *ws, size_t ws_bytes,
                                        hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(count >= 0 && N >= 0, DP_EINVAL);
    DPG_REQUIRE(count == 0 || params != nullptr, DP_EINVAL);
    DPG_REQUIRE(C > 0.0f && sigma >= 0.0f && denom > 0.0f, DP_EINVAL);
    DPG_REQUIRE(!(sigma > 0.0f && __builtin_isinf(C)), DP_EINVAL);
    bool any_col = false;
    for (int i = 0; i < count; ++i) {
        const dp_param &q = params[i];
        DPG_REQUIRE(q.numel >= 0 && (q.flags & ~(uint32_t)DP_PARAM_REDUCE) == 0, DP_EINVAL);
        DPG_REQUIRE(q.numel / 4 < (i64(1) << 32), DP_EINVAL);
        DPG_REQUIRE(q.numel == 0 || q.sum != nullptr, DP_EINVAL);
        if (q.flags & DP_PARAM_REDUCE) {
            DPG_REQUIRE(N == 0 || q.numel == 0 || q.grad_sample != nullptr, DP_EINVAL);
            any_col = true;
        }
    }
    DPG_REQUIRE(!any_col || N == 0 || norm != nullptr, DP_EINVAL);
    const size_t need = dp_clip_noise_many_workspace_bytes(params, count, N);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    const bool noise = sigma > 0.0f;
    const float sc = noise ? sigma * C : 0.0f;
    for (int first = 0; first < count; first += kMaxGroup) {
        const int c = count - first < kMaxGroup ? count - first : kMaxGroup;
        GroupDesc d;
        describe(params, first, c, N, d);
        if (d.cblocks > 0)
            colsum_many_kernel<<<(unsigned)(d.cblocks * d.splits), kThreads, 0, stream>>>(d, norm, C, (float *)ws);
        if (d.fblocks > 0)
            finish_many_kernel<<<(unsigned)d.fblocks, kThreads, 0, stream>>>(
                d, (const float *)ws, (uint32_t)seed, (uint32_t)(seed >> 32), step, step_dev, sc, denom,
                noise ? 1 : 0);
    }
    return launch_status();
}

extern "C" dp_status dp_step_advance(uint64_t *step_dev, uint64_t by, hipStream_t stream)
{
    DPG_REQUIRE(step_dev != nullptr, DP_EINVAL);
    step_advance_kernel<<<1, 64, 0, stream>>>(step_dev, by);
    return launch_status();
}
