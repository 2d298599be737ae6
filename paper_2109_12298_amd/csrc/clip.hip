// Per-sample norms, clip factors and clipped sums (the DP-SGD step of the
// paper's section 1: clip each per-sample gradient's l2 norm, then add the
// clipped gradients over the batch).
//
// All reductions run in a fixed order: samples ascending for the clipped
// sums, layers ascending for the norms.  The column reduction splits the
// batch into contiguous sample ranges when a tensor is too small to fill the
// GPU; the range partials are then added in range order.
#include "common.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;

__global__ void norms_kernel(const float *__restrict__ sq, int L, i64 N, float *__restrict__ norm,
                             int32_t *status)
{
    const i64 n = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    float s = 0.0f;
    s = ordered_sum(sq + n, N, L);
    const float r = sqrtf(s);
    if (!isfinite(r)) raise_flag(status, DP_FLAG_NONFINITE);
    norm[n] = r;
}

__global__ void clip_factors_kernel(const float *__restrict__ norm, i64 N, float C,
                                    float *__restrict__ c, int32_t *status)
{
    const i64 n = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    const float x = norm[n];
    if (!isfinite(x)) raise_flag(status, DP_FLAG_NONFINITE);
    c[n] = clip_factor(x, C);
}

template <bool VEC>
__global__ __launch_bounds__(kThreads) void sqnorm_rows_kernel(const float *__restrict__ G,
                                                               i64 numel,
                                                               float *__restrict__ sqnorm)
{
    __shared__ float red[16];
    const i64 n = blockIdx.x;
    const float *g = G + n * numel;
    float s = 0.0f;
    if (VEC && (numel & 3) == 0) {
        const float4 *g4 = reinterpret_cast<const float4 *>(g);
        for (i64 i = threadIdx.x; i < numel / 4; i += kThreads) {
            const float4 v = g4[i];
            s += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
        }
    } else {
        for (i64 i = threadIdx.x; i < numel; i += kThreads) s += g[i] * g[i];
    }
    s = block_sum(s, red);
    if (threadIdx.x == 0) sqnorm[n] = s;
}

// sum[e] (or part[split][e]) = sum over the split's samples of c_n * G[n][e].
template <bool VEC>
__global__ __launch_bounds__(kThreads) void colsum_kernel(const float *__restrict__ G,
                                                          const float *__restrict__ norm, float C,
                                                          i64 N, i64 numel, i64 per_split,
                                                          int eblocks, float *__restrict__ out)
{
    const int split = blockIdx.x / eblocks;
    const int eb = blockIdx.x % eblocks;
    const i64 n0 = (i64)split * per_split;
    const i64 n1 = n0 + per_split < N ? n0 + per_split : N;
    float *o = out + (i64)split * numel;
    if (VEC) {
        const i64 e4 = (i64)eb * kThreads + threadIdx.x;
        if (4 * e4 >= numel) return;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        const float4 *g = reinterpret_cast<const float4 *>(G) + e4;
        const i64 stride = numel / 4;
        i64 n = n0;
        for (; n + 4 <= n1; n += 4) {
            const float4 a0 = g[(n + 0) * stride], a1 = g[(n + 1) * stride];
            const float4 a2 = g[(n + 2) * stride], a3 = g[(n + 3) * stride];
            const float c0 = clip_factor(norm[n + 0], C), c1 = clip_factor(norm[n + 1], C);
            const float c2 = clip_factor(norm[n + 2], C), c3 = clip_factor(norm[n + 3], C);
            acc.x += c0 * a0.x; acc.y += c0 * a0.y; acc.z += c0 * a0.z; acc.w += c0 * a0.w;
            acc.x += c1 * a1.x; acc.y += c1 * a1.y; acc.z += c1 * a1.z; acc.w += c1 * a1.w;
            acc.x += c2 * a2.x; acc.y += c2 * a2.y; acc.z += c2 * a2.z; acc.w += c2 * a2.w;
            acc.x += c3 * a3.x; acc.y += c3 * a3.y; acc.z += c3 * a3.z; acc.w += c3 * a3.w;
        }
        for (; n < n1; ++n) {
            const float4 a = g[n * stride];
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

__global__ void range_sum_kernel(const float *__restrict__ part, int splits, i64 count,
                                 float *__restrict__ out)
{
    const i64 e = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count) return;
    float s = 0.0f;
    s = ordered_sum(part + e, count, splits);
    out[e] = s;
}

struct ColSplit {
    int eblocks, splits;
    i64 per_split;
    bool vec;
};

ColSplit col_split(i64 N, i64 numel, bool vec_ok)
{
    ColSplit s;
    s.vec = (numel & 3) == 0 && vec_ok;
    const i64 per_block = s.vec ? 4 * kThreads : kThreads;
    s.eblocks = (int)ceil_div(numel, per_block);
    i64 want = ceil_div(2048, s.eblocks);
    const i64 max_splits = N / 16;                 // keep at least 16 samples per range
    if (want > max_splits) want = max_splits;
    if (want > 64) want = 64;
    if (want < 1) want = 1;
    s.per_split = N > 0 ? ceil_div(N, want) : 1;
    s.splits = N > 0 ? (int)ceil_div(N, s.per_split) : 1;
    return s;
}

// One wave per embedding row v.  Lane l binary-searches sample (n0 + l)'s
// sorted ids for v; the hits are then visited in ascending sample order.
constexpr int kEmbR = 4;   // columns per lane per pass: the wave covers 256 columns

__global__ __launch_bounds__(kThreads) void emb_clipsum_kernel(
    const int64_t *__restrict__ row_ptr, const int64_t *__restrict__ uniq,
    const float *__restrict__ rows, const float *__restrict__ norm, float C, i64 N, i64 V, i64 D,
    float *__restrict__ sum, int32_t *status)
{
    const int lane = threadIdx.x & 63;
    const i64 gtid = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    const i64 nthreads = (i64)gridDim.x * blockDim.x;
    // stored ids outside [0, V) are reported and never matched
    const i64 nnz = row_ptr[N];
    for (i64 e = gtid; e < nnz; e += nthreads)
        if (uniq[e] < 0 || uniq[e] >= V) raise_flag(status, DP_FLAG_BAD_INDEX);

    const i64 v = (i64)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (v >= V) return;
    for (i64 d0 = 0; d0 < D; d0 += 64 * kEmbR) {
        float acc[kEmbR];
#pragma unroll
        for (int q = 0; q < kEmbR; ++q) acc[q] = 0.0f;
        for (i64 nc = 0; nc < N; nc += 64) {
            const i64 n = nc + lane;
            i64 hit = -1;
            if (n < N) {
                i64 lo = row_ptr[n], hi = row_ptr[n + 1];
                while (lo < hi) {
                    const i64 mid = lo + ((hi - lo) >> 1);
                    if (uniq[mid] < v) lo = mid + 1;
                    else hi = mid;
                }
                if (lo < row_ptr[n + 1] && uniq[lo] == v) hit = lo;
            }
            uint64_t mask = __ballot(hit >= 0);
            while (mask) {
                const int b = __ffsll((unsigned long long)mask) - 1;
                mask &= mask - 1;
                const i64 k = __shfl(hit, b, 64);
                const float cn = clip_factor(norm[nc + b], C);
#pragma unroll
                for (int q = 0; q < kEmbR; ++q) {
                    const i64 d = d0 + lane + 64 * q;
                    if (d < D) acc[q] += cn * rows[k * D + d];
                }
            }
        }
#pragma unroll
        for (int q = 0; q < kEmbR; ++q) {
            const i64 d = d0 + lane + 64 * q;
            if (d < D) sum[v * D + d] = acc[q];
        }
    }
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" dp_status dp_per_sample_norms(const float *sqnorm, int32_t n_layers, int64_t N,
                                         float *norm, int32_t *status, hipStream_t stream)
{
    DPG_REQUIRE(n_layers >= 0 && N >= 0, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (norm != nullptr && (n_layers == 0 || sqnorm != nullptr)), DP_EINVAL);
    if (N == 0) return DP_OK;
    norms_kernel<<<(unsigned)ceil_div(N, 256), 256, 0, stream>>>(sqnorm, n_layers, N, norm, status);
    return launch_status();
}

extern "C" dp_status dp_sqnorm_from_grads(const float *G, int64_t N, int64_t numel, float *sqnorm,
                                          int32_t *status, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(N >= 0 && numel >= 0, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (sqnorm != nullptr && (numel == 0 || G != nullptr)), DP_EINVAL);
    if (N == 0) return DP_OK;
    if (aligned(G, 16))
        sqnorm_rows_kernel<true><<<(unsigned)N, kThreads, 0, stream>>>(G, numel, sqnorm);
    else
        sqnorm_rows_kernel<false><<<(unsigned)N, kThreads, 0, stream>>>(G, numel, sqnorm);
    return launch_status();
}

extern "C" dp_status dp_clip_factors(const float *norm, int64_t N, float C, float *c,
                                     int32_t *status, hipStream_t stream)
{
    DPG_REQUIRE(N >= 0 && C > 0.0f, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (norm != nullptr && c != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;
    clip_factors_kernel<<<(unsigned)ceil_div(N, 256), 256, 0, stream>>>(norm, N, C, c, status);
    return launch_status();
}

extern "C" size_t dp_clip_accumulate_workspace_bytes(int64_t N, int64_t numel)
{
    if (N <= 0 || numel <= 0) return 0;
    // the split never depends on pointer alignment: query with the vector layout
    const ColSplit s = col_split(N, numel, true);
    return s.splits > 1 ? (size_t)s.splits * (size_t)numel * sizeof(float) : 0;
}

extern "C" dp_status dp_clip_accumulate(const float *G, const float *norm, float C, int64_t N,
                                        int64_t numel, float *sum, float *c_out, int32_t *status,
                                        void *ws, size_t ws_bytes, hipStream_t stream)
{
    DPG_REQUIRE(N >= 0 && numel >= 0 && C > 0.0f, DP_EINVAL);
    DPG_REQUIRE(numel == 0 || sum != nullptr, DP_EINVAL);
    DPG_REQUIRE(N == 0 || norm != nullptr, DP_EINVAL);
    DPG_REQUIRE(N == 0 || numel == 0 || G != nullptr, DP_EINVAL);
    const size_t need = dp_clip_accumulate_workspace_bytes(N, numel);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (c_out && N > 0)
        clip_factors_kernel<<<(unsigned)ceil_div(N, 256), 256, 0, stream>>>(norm, N, C, c_out, status);
    if (numel == 0) return launch_status();
    if (N == 0) {
        zero_fill(sum, numel, stream);
        return launch_status();
    }
    ColSplit s = col_split(N, numel, true);
    float *dst = s.splits > 1 ? (float *)ws : sum;
    s.vec = s.vec && aligned(G, 16) && aligned(dst, 16);
    if (!s.vec) s.eblocks = (int)ceil_div(numel, kThreads);
    const dim3 grid((unsigned)(s.splits * s.eblocks));
    if (s.vec)
        colsum_kernel<true><<<grid, kThreads, 0, stream>>>(G, norm, C, N, numel, s.per_split, s.eblocks, dst);
    else
        colsum_kernel<false><<<grid, kThreads, 0, stream>>>(G, norm, C, N, numel, s.per_split, s.eblocks, dst);
    if (s.splits > 1)
        range_sum_kernel<<<(unsigned)ceil_div(numel, 256), 256, 0, stream>>>(dst, s.splits, numel, sum);
    return launch_status();
}

extern "C" dp_status dp_clip_accumulate_embedding(const int64_t *row_ptr, const int64_t *uniq_ids,
                                                  const float *rows, const float *norm, float C,
                                                  int64_t N, int64_t V, int64_t D, float *sum,
                                                  int32_t *status, hipStream_t stream)
{
    DPG_REQUIRE(N >= 0 && V >= 1 && D >= 1 && C > 0.0f, DP_EINVAL);
    DPG_REQUIRE(row_ptr != nullptr && sum != nullptr, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (norm != nullptr && uniq_ids != nullptr && rows != nullptr), DP_EINVAL);
    const unsigned blocks = (unsigned)ceil_div(V, kThreads / 64);
    emb_clipsum_kernel<<<blocks, kThreads, 0, stream>>>(row_ptr, uniq_ids, rows, norm, C, N, V, D,
                                                        sum, status);
    return launch_status();
}
