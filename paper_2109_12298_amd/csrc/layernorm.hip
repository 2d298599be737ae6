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

// ---------------------------------------------------------------------------
// Several layers in one launch (dp_grad_sample_layernorm_many).  A workgroup
// owns one (layer, sample, chunk of 128 bytes of features: 64 bf16 or 32
// fp32) and adds every position itself, so nothing but one squared-norm
// partial per (sample, chunk) goes through memory: thread i takes the
// 16-byte piece i % 8 of rows i / 8, i / 8 + 32, ... (ascending t), the 32
// row groups' sums are then added in row-group order through LDS, and the
// features' gradients are written directly.  A second launch adds each
// sample's chunk partials in chunk order.
// ---------------------------------------------------------------------------
constexpr int kLnGroupMax = 16;
constexpr int kLnRowGroups = kThreads / 8;            // rows in flight per pass

struct LnLayer {
    const void *xh, *B;
    float *gg, *gb, *part, *sqnorm;
    i64 T, D;
    int chunks, blk0;
    float scale;
};

struct LnGroup {
    i64 N;
    int count;
    LnLayer L[kLnGroupMax];
};

// 16 bytes of a row as fp32: eight bf16 or four fp32 features
template <typename T>
struct Piece;

template <>
struct Piece<uint16_t> {
    static constexpr int E = 8;
    __device__ static void load(const uint16_t *p, float (&v)[8])
    {
        const uint4 u = *reinterpret_cast<const uint4 *>(p);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[2 * i] = __uint_as_float(w[i] << 16);
            v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
};

template <>
struct Piece<float> {
    static constexpr int E = 4;
    __device__ static void load(const float *p, float (&v)[4])
    {
        const float4 u = *reinterpret_cast<const float4 *>(p);
        v[0] = u.x; v[1] = u.y; v[2] = u.z; v[3] = u.w;
    }
};

// VEC: D a multiple of the piece and 16-byte aligned rows (one 16-byte load
// per piece); else element loads, bounds-checked
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void ln_rows_group_kernel(const LnGroup g)
{
    constexpr int E = Piece<T>::E;
    constexpr int F = 8 * E;                           // features per chunk
    __shared__ float red[2][kLnRowGroups][F + 1];
    __shared__ float wsq[kThreads / kWave];
    const int b = (int)blockIdx.x;
    int k = 0;
    while (k + 1 < g.count && g.L[k + 1].blk0 <= b) ++k;
    const LnLayer &L = g.L[k];
    const int l = b - L.blk0;
    const i64 n = l / L.chunks;
    const int ch = l % L.chunks;
    const int tid = threadIdx.x, lane = tid & 63;
    const int rg = tid >> 3, pc = tid & 7;
    const i64 Tn = L.T, D = L.D;
    const i64 f0 = (i64)ch * F + pc * E;               // this thread's first feature
    const T *xh = reinterpret_cast<const T *>(L.xh) + n * Tn * D + f0;
    const T *Bp = reinterpret_cast<const T *>(L.B) + n * Tn * D + f0;
    float ag[E], ab[E];
#pragma unroll
    for (int e = 0; e < E; ++e) ag[e] = ab[e] = 0.0f;
    auto add = [&](const float (&bv)[E], const float (&xv)[E]) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            ag[e] += bv[e] * xv[e];
            ab[e] += bv[e];
        }
    };
    if (VEC ? f0 < D : true) {
        i64 t = rg;
        // four passes' loads in flight, rows still added in ascending t
        for (; t + 3 * kLnRowGroups < Tn; t += 4 * kLnRowGroups) {
            float bv[4][E], xv[4][E];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const i64 o = (t + q * kLnRowGroups) * D;
                if constexpr (VEC) {
                    Piece<T>::load(Bp + o, bv[q]);
                    Piece<T>::load(xh + o, xv[q]);
                } else {
#pragma unroll
                    for (int e = 0; e < E; ++e) {
                        const bool in = f0 + e < D;
                        bv[q][e] = in ? load_elem<T>(Bp, o + e) : 0.0f;
                        xv[q][e] = in ? load_elem<T>(xh, o + e) : 0.0f;
                    }
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) add(bv[q], xv[q]);
        }
        for (; t < Tn; t += kLnRowGroups) {
            float bv[E], xv[E];
            const i64 o = t * D;
            if constexpr (VEC) {
                Piece<T>::load(Bp + o, bv);
                Piece<T>::load(xh + o, xv);
            } else {
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    const bool in = f0 + e < D;
                    bv[e] = in ? load_elem<T>(Bp, o + e) : 0.0f;
                    xv[e] = in ? load_elem<T>(xh, o + e) : 0.0f;
                }
            }
            add(bv, xv);
        }
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
        red[0][rg][pc * E + e] = ag[e];
        red[1][rg][pc * E + e] = ab[e];
    }
    __syncthreads();
    // thread i < 2 F: feature i % F of gamma (i < F) or beta, row groups in order
    float sq = 0.0f;
    if (tid < 2 * F) {
        const int h = tid / F, f = tid % F;
        float s = 0.0f;
        for (int r = 0; r < kLnRowGroups; ++r) s += red[h][r][f];
        s *= L.scale;
        const i64 col = (i64)ch * F + f;
        if (col < D) {
            (h == 0 ? L.gg : L.gb)[n * D + col] = s;
            sq = s * s;
        }
    }
    sq = wave_sum(sq);
    if (lane == 0) wsq[tid >> 6] = sq;
    __syncthreads();
    if (tid == 0 && L.sqnorm) {
        float t = 0.0f;
        for (int w = 0; w < kThreads / kWave; ++w) t += wsq[w];
        (L.chunks > 1 ? L.part[n * L.chunks + ch] : L.sqnorm[n]) = t;
    }
}

// sqnorm[n] of each layer with several chunks: one wave per (layer, sample)
// adds the chunk partials (lane l takes l, l + 64, ..., then a butterfly)
__global__ __launch_bounds__(256) void ln_chunk_sum_kernel(const LnGroup g)
{
    const LnLayer &L = g.L[blockIdx.y];
    const i64 n = (i64)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (L.chunks == 1 || L.sqnorm == nullptr || n >= g.N) return;
    const float *q = L.part + n * L.chunks;
    float s = 0.0f;
    for (int c = lane; c < L.chunks; c += kWave) s += q[c];
    s = wave_sum(s);
    if (lane == 0) L.sqnorm[n] = s;
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

extern "C" size_t dp_grad_sample_layernorm_many_workspace_bytes(const dp_layernorm_layer *items, int32_t count,
                                                                int64_t N, dp_dtype dt)
{
    if (items == nullptr || count <= 0 || N <= 0 || !dtype_ok(dt)) return 0;
    const i64 F = 128 / (i64)dtype_bytes(dt);
    size_t b = 0;
    for (int i = 0; i < count; ++i) {
        const i64 chunks = items[i].D > 0 ? ceil_div(items[i].D, F) : 1;
        if (chunks > 1) b += (size_t)((N * chunks * (i64)sizeof(float) + 255) & ~i64(255));
    }
    return b;
}

extern "C" dp_status dp_grad_sample_layernorm_many(const dp_layernorm_layer *items, int32_t count, dp_dtype dt,
                                                   int64_t N, int32_t *status, void *ws, size_t ws_bytes,
                                                   hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(count >= 0 && count <= 64 && (count == 0 || items != nullptr), DP_EINVAL);
    DPG_REQUIRE(N >= 0 && N < (i64(1) << 31), DP_EINVAL);
    for (int i = 0; i < count; ++i) {
        const dp_layernorm_layer &it = items[i];
        DPG_REQUIRE(it.T >= 0 && it.D >= 1, DP_EINVAL);
        DPG_REQUIRE(N == 0 || (it.ggamma != nullptr && it.gbeta != nullptr), DP_EINVAL);
        DPG_REQUIRE(N * it.T == 0 || (it.xhat != nullptr && it.B != nullptr), DP_EINVAL);
    }
    const size_t need = dp_grad_sample_layernorm_many_workspace_bytes(items, count, N, dt);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0 || count == 0) return DP_OK;
    const i64 F = 128 / (i64)dtype_bytes(dt);
    const i64 pc = 16 / (i64)dtype_bytes(dt);
    char *w = (char *)ws;
    LnLayer lay[64];
    bool vec[64];
    for (int i = 0; i < count; ++i) {
        const dp_layernorm_layer &it = items[i];
        LnLayer &L = lay[i];
        L.xh = it.xhat;
        L.B = it.B;
        L.gg = it.ggamma;
        L.gb = it.gbeta;
        L.sqnorm = it.sqnorm;
        L.T = it.T;
        L.D = it.D;
        L.scale = it.scale;
        L.chunks = (int)ceil_div(it.D, F);
        L.part = nullptr;
        if (L.chunks > 1) {
            L.part = (float *)w;
            w += (N * L.chunks * (i64)sizeof(float) + 255) & ~i64(255);
        }
        vec[i] = it.D % pc == 0 && aligned(it.xhat, 16) && aligned(it.B, 16);
    }
    // the rows launches: the 16-byte class, then the element class
    for (int cls = 0; cls < 2; ++cls) {
        LnGroup g;
        g.N = N;
        g.count = 0;
        i64 blocks = 0;
        for (int i = 0; i <= count; ++i) {
            if (i < count && vec[i] == (cls == 0)) {
                lay[i].blk0 = (int)blocks;
                blocks += N * lay[i].chunks;
                DPG_REQUIRE(blocks < (i64(1) << 31), DP_EUNSUPPORTED);
                g.L[g.count++] = lay[i];
            }
            if (g.count > 0 && (g.count == kLnGroupMax || i == count)) {
                const unsigned grid = (unsigned)blocks;
                if (dt == DP_BF16) {
                    if (cls == 0) ln_rows_group_kernel<uint16_t, true><<<grid, kThreads, 0, stream>>>(g);
                    else ln_rows_group_kernel<uint16_t, false><<<grid, kThreads, 0, stream>>>(g);
                } else {
                    if (cls == 0) ln_rows_group_kernel<float, true><<<grid, kThreads, 0, stream>>>(g);
                    else ln_rows_group_kernel<float, false><<<grid, kThreads, 0, stream>>>(g);
                }
                g.count = 0;
                blocks = 0;
            }
        }
    }
    // several chunks: add each sample's chunk partials
    {
        LnGroup g;
        g.N = N;
        g.count = 0;
        for (int i = 0; i <= count; ++i) {
            if (i < count && lay[i].chunks > 1 && lay[i].sqnorm) g.L[g.count++] = lay[i];
            if (g.count > 0 && (g.count == kLnGroupMax || i == count)) {
                ln_chunk_sum_kernel<<<dim3((unsigned)ceil_div(N, 4), (unsigned)g.count), 256, 0, stream>>>(g);
                g.count = 0;
            }
        }
    }
    return launch_status();
}
