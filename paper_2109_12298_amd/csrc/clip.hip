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

// n_active (device, may be null): samples n >= *n_active are outside the
// batch and get the norm -1 (clip factor 0), without a flag.
__global__ void norms_kernel(const float *__restrict__ sq, int L, i64 N, const int64_t *n_active,
                             float *__restrict__ norm, int32_t *status)
{
    const i64 n = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    if (n_active && n >= *n_active) {
        norm[n] = -1.0f;
        return;
    }
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

// Embedding clipped sum over CSR rows, 64 samples (one wave's lanes) at a
// time.  The chunk's CSR is inverted into a dense map [V][64] of row indices
// (-1 where a sample does not hold id v): a fill, then one scatter per stored
// row.  A wave per id v then reads its 64 map entries with one coalesced load
// and adds the hit rows in ascending sample order, eight rows' loads in flight
// at a time, onto the previous chunks' sum.
constexpr int kChunk = 64;
constexpr int kEmbBatch = 8;

__global__ void emb_map_fill_kernel(int32_t *__restrict__ map, i64 n4)
{
    const i64 i = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n4) reinterpret_cast<int4 *>(map)[i] = make_int4(-1, -1, -1, -1);
}

// one workgroup per sample of the chunk: map[uniq[k]][n - n0] = k
__global__ __launch_bounds__(kThreads) void emb_map_scatter_kernel(
    const int64_t *__restrict__ row_ptr, const int64_t *__restrict__ uniq, i64 n0, i64 V, i64 cap,
    int32_t *__restrict__ map, int32_t *status)
{
    const i64 n = n0 + blockIdx.x;
    const i64 lo = row_ptr[n], hi = row_ptr[n + 1];
    if (hi > cap && threadIdx.x == 0) raise_flag(status, DP_FLAG_CAP);
    const i64 end = hi < cap ? hi : cap;
    for (i64 k = lo + threadIdx.x; k < end; k += kThreads) {
        const int64_t v = uniq[k];
        if (v < 0 || v >= V) raise_flag(status, DP_FLAG_BAD_INDEX);
        else map[v * kChunk + blockIdx.x] = (int32_t)k;
    }
}

template <int VEC>
__global__ __launch_bounds__(kThreads) void emb_clipsum_kernel(
    const int32_t *__restrict__ map, const float *__restrict__ rows, const float *__restrict__ norm, float C,
    i64 n0, int nc, i64 V, i64 D, int first, float *__restrict__ sum)
{
    const int lane = threadIdx.x & 63;
    const i64 v = (i64)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (v >= V) return;
    const int hit = lane < nc ? map[v * kChunk + lane] : -1;
    const float cn = lane < nc ? clip_factor(norm[n0 + lane], C) : 0.0f;
    const uint64_t all = __ballot(hit >= 0);
    for (i64 c0 = 0; c0 < D; c0 += 64 * VEC) {
        const i64 c = c0 + (i64)VEC * lane;
        const bool on = c < D;
        const i64 cc = on ? c : 0;
        float acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0f;
        if (!first && on) {
            if constexpr (VEC == 4) {
                const float4 q = *reinterpret_cast<const float4 *>(sum + v * D + c);
                acc[0] = q.x; acc[1] = q.y; acc[2] = q.z; acc[3] = q.w;
            } else {
                acc[0] = sum[v * D + c];
            }
        }
        // batches of the hit lanes in ascending order; slots past the last
        // hit repeat the first (a valid row) and are not added
        const int first_hit = all ? __ffsll((unsigned long long)all) - 1 : 0;
        uint64_t mask = all;
        while (mask) {
            int kk[kEmbBatch];
            float cj[kEmbBatch];
            bool ok[kEmbBatch];
#pragma unroll
            for (int j = 0; j < kEmbBatch; ++j) {
                ok[j] = mask != 0;
                const int b = ok[j] ? __ffsll((unsigned long long)mask) - 1 : first_hit;
                mask &= mask - 1;
                kk[j] = __shfl(hit, b, 64);
                cj[j] = __shfl(cn, b, 64);
            }
            float x[kEmbBatch][VEC];
#pragma unroll
            for (int j = 0; j < kEmbBatch; ++j) {
                const float *src = rows + (i64)kk[j] * D + cc;
                if constexpr (VEC == 4) {
                    const float4 q = *reinterpret_cast<const float4 *>(src);
                    x[j][0] = q.x; x[j][1] = q.y; x[j][2] = q.z; x[j][3] = q.w;
                } else {
                    x[j][0] = src[0];
                }
            }
#pragma unroll
            for (int j = 0; j < kEmbBatch; ++j)
                if (ok[j])
#pragma unroll
                    for (int i = 0; i < VEC; ++i) acc[i] += cj[j] * x[j][i];
        }
        if (on) {
            if constexpr (VEC == 4)
                *reinterpret_cast<float4 *>(sum + v * D + c) = make_float4(acc[0], acc[1], acc[2], acc[3]);
            else
                sum[v * D + c] = acc[0];
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
    norms_kernel<<<(unsigned)ceil_div(N, 256), 256, 0, stream>>>(sqnorm, n_layers, N, nullptr, norm, status);
    return launch_status();
}

extern "C" dp_status dp_per_sample_norms_active(const float *sqnorm, int32_t n_layers, int64_t N,
                                                const int64_t *n_active, float *norm, int32_t *status,
                                                hipStream_t stream)
{
    DPG_REQUIRE(n_layers >= 0 && N >= 0, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (norm != nullptr && (n_layers == 0 || sqnorm != nullptr)), DP_EINVAL);
    if (N == 0) return DP_OK;
    norms_kernel<<<(unsigned)ceil_div(N, 256), 256, 0, stream>>>(sqnorm, n_layers, N, n_active, norm, status);
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

extern "C" size_t dp_clip_accumulate_embedding_workspace_bytes(int64_t N, int64_t V)
{
    if (N <= 0 || V <= 0) return 0;
    return (size_t)V * kChunk * sizeof(int32_t);
}

extern "C" dp_status dp_clip_accumulate_embedding(const int64_t *row_ptr, const int64_t *uniq_ids,
                                                  const float *rows, int64_t cap, const float *norm, float C,
                                                  int64_t N, int64_t V, int64_t D, float *sum,
                                                  int32_t *status, void *ws, size_t ws_bytes,
                                                  hipStream_t stream)
{
    DPG_REQUIRE(N >= 0 && V >= 1 && D >= 1 && cap >= 0 && C > 0.0f, DP_EINVAL);
    DPG_REQUIRE(V < (i64(1) << 31) / kChunk, DP_EUNSUPPORTED);
    DPG_REQUIRE(row_ptr != nullptr && sum != nullptr, DP_EINVAL);
    DPG_REQUIRE(N == 0 || norm != nullptr, DP_EINVAL);
    DPG_REQUIRE(cap == 0 || (uniq_ids != nullptr && rows != nullptr), DP_EINVAL);
    DPG_REQUIRE(cap < (i64(1) << 31), DP_EUNSUPPORTED);
    const size_t need = dp_clip_accumulate_embedding_workspace_bytes(N, V);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    DPG_REQUIRE(need == 0 || aligned(ws, 16), DP_EINVAL);
    if (N == 0) {
        zero_fill(sum, V * D, stream);
        return launch_status();
    }
    int32_t *map = (int32_t *)ws;
    const i64 n4 = V * kChunk / 4;
    const bool vec = D % 4 == 0 && aligned(rows, 16) && aligned(sum, 16);
    const unsigned vblocks = (unsigned)ceil_div(V, kThreads / 64);
    for (i64 n0 = 0; n0 < N; n0 += kChunk) {
        const int nc = (int)(N - n0 < kChunk ? N - n0 : kChunk);
        emb_map_fill_kernel<<<(unsigned)ceil_div(n4, kThreads), kThreads, 0, stream>>>(map, n4);
        emb_map_scatter_kernel<<<(unsigned)nc, kThreads, 0, stream>>>(row_ptr, uniq_ids, n0, V, cap, map,
                                                                       status);
        if (vec)
            emb_clipsum_kernel<4><<<vblocks, kThreads, 0, stream>>>(map, rows, norm, C, n0, nc, V, D, n0 == 0,
                                                                    sum);
        else
            emb_clipsum_kernel<1><<<vblocks, kThreads, 0, stream>>>(map, rows, norm, C, n0, nc, V, D, n0 == 0,
                                                                    sum);
    }
    return launch_status();
}
