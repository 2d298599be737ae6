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
    float *Acc[kMaxGroup];         // running sum over the physical batches of a logical one, or null
    i64 numel[kMaxGroup];
    i64 ws_off[kMaxGroup];         // first partial of the tensor, in floats
    i64 stride[kMaxGroup];         // floats between two ranges' partials of the tensor
    int cblk0[kMaxGroup + 1];      // first column-reduce workgroup of each tensor
    int fblk0[kMaxGroup + 1];      // first finish workgroup of each tensor
    uint32_t pidx[kMaxGroup];
    uint32_t flags[kMaxGroup];     // bit 0: column-reduce vectorized, bit 1: finish vectorized,
                                   // bit 2: the sum S is read in 16-byte pieces
    uint8_t R[kMaxGroup];          // 1: the tensor's sum is formed here from per-sample grads
};

// with a running sum: acc += s, and s becomes the running sum (what the
// output is formed from)
__device__ __forceinline__ void accumulate(float *acc, i64 e0, int cnt, float (&s)[4])
{
    if (acc == nullptr) return;
    for (int i = 0; i < cnt; ++i) {
        s[i] += acc[e0 + i];
        acc[e0 + i] = s[i];
    }
}

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
    } else if (cnt == 4 && (d.flags[p] & 4u)) {
        const float4 v = reinterpret_cast<const float4 *>(d.S[p])[e0 / 4];
        s[0] = v.x; s[1] = v.y; s[2] = v.z; s[3] = v.w;
    } else {
        for (int i = 0; i < cnt; ++i) s[i] = d.S[p][e0 + i];
    }
    if (col && (from_parts || d.N == 0)) {
        for (int i = 0; i < cnt; ++i) d.S[p][e0 + i] = s[i];
    }
    accumulate(d.Acc[p], e0, cnt, s);
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

// ---------------------------------------------------------------------------
// One-launch variant: norms (optional), column reduce, and finish.
//
// A column workgroup owns 256 / KG float4 columns of a column-reduced tensor
// (scalar columns when the tensor is not 16-byte vectorizable) for the whole
// batch: its 256 threads are KG sample groups x 256 / KG columns, each group
// adding c_n * G[n] over a contiguous range of ceil(N / KG) samples in
// ascending n.  The KG range sums are then added in range order through LDS,
// so the clipped sum is deterministic without a
// second launch or any communication between workgroups, and the same
// workgroup adds the noise and divides.  Blocks past the column work finish
// the tensors whose sums were formed elsewhere.  With sqnorm given, every
// workgroup computes the clip factors of the batch from the layers' squared
// norms (added in layer order, as norms_kernel does) and workgroup 0 writes
// the norms.
// ---------------------------------------------------------------------------
// A column workgroup splits the batch into KG sample groups (4, 8 or 16) and
// covers kThreads / KG columns: fewer groups give longer contiguous rows per
// load, more groups give more workgroups; the launch takes the fewest groups
// that still give every CU a column workgroup.
constexpr int kMinColBlocks = 256;
constexpr int kCfChunk = 4096;              // clip factors held in LDS at a time

struct FusedArgs {
    const float *sqnorm;       // [L][N] or null (then norm is an input)
    int L;
    float *norm;               // [N]: written from sqnorm, else read
    float C;
    uint32_t k0, k1;
    uint64_t step;
    const uint64_t *step_dev;
    float sc, denom;
    int noise;
    // noise schedule: sigma of step t is sigma_tab[min(t, tab_len - 1)]
    // (then sc = sigma * C and noise = sigma > 0 are taken at run time)
    const float *sigma_tab;
    i64 tab_len;
    // active batch (device, may be null): samples n >= *n_active are padding,
    // left out of the sums, their norms set to -1 when computed here
    const int64_t *n_active;
    int32_t *status;
    int cblocks;               // column workgroups
    int cblk0[kMaxGroup + 1];  // first column workgroup of each tensor
    int oblk0[kMaxGroup + 1];  // first finish-only workgroup of each tensor
};

static_assert(sizeof(GroupDesc) + sizeof(FusedArgs) <= 4096, "kernel arguments");

// The noise scale sigma * C of this launch's step, and whether to draw noise:
// fixed, or the step's entry of the schedule (a negative or non-finite entry
// raises DP_FLAG_NONFINITE and gives a NaN scale).
__device__ __forceinline__ void noise_scale(const FusedArgs &f, float &sc, bool &noise)
{
    if (f.sigma_tab == nullptr) {
        sc = f.sc;
        noise = f.noise != 0;
        return;
    }
    const uint64_t t = f.step + (f.step_dev ? *f.step_dev : 0ull);
    const uint64_t last = (uint64_t)(f.tab_len - 1);
    const float sg = f.sigma_tab[t < last ? t : last];
    if (!(sg >= 0.0f) || !isfinite(sg)) {
        if (threadIdx.x == 0) raise_flag(f.status, DP_FLAG_NONFINITE);
        sc = __builtin_nanf("");
        noise = true;
        return;
    }
    sc = sg * f.C;
    noise = sg > 0.0f;
}

// STREAM: the per-sample gradients are read with non-temporal loads (they
// are read once, and a large set of them would only push out of the caches
// what the next kernels read).
template <bool STREAM, int KG>
__global__ __launch_bounds__(kThreads) void norms_clip_noise_kernel(GroupDesc d, FusedArgs f)
{
    constexpr int kCols = kThreads / KG;
    __shared__ float cfs[kCfChunk];
    __shared__ float4 part[KG][kCols];
    const int tid = threadIdx.x;
    if ((int)blockIdx.x >= f.cblocks) {
        // finish-only: a tensor whose sum is already in S (or an empty batch)
        const int b = (int)blockIdx.x - f.cblocks;
        const int p = find_param(f.oblk0, d.count, b);
        const i64 numel = d.numel[p];
        const i64 q = (i64)(b - f.oblk0[p]) * kThreads + tid;
        const i64 e0 = 4 * q;
        if (e0 >= numel) return;
        const int cnt = e0 + 4 <= numel ? 4 : (int)(numel - e0);
        float s[4] = {0.f, 0.f, 0.f, 0.f};
        if (d.R[p]) {
            for (int i = 0; i < cnt; ++i) d.S[p][e0 + i] = 0.0f;   // N = 0: the clipped sum is zero
        } else if (cnt == 4 && (d.flags[p] & 4u)) {
            const float4 v = reinterpret_cast<const float4 *>(d.S[p])[q];
            s[0] = v.x; s[1] = v.y; s[2] = v.z; s[3] = v.w;
        } else {
            for (int i = 0; i < cnt; ++i) s[i] = d.S[p][e0 + i];
        }
        accumulate(d.Acc[p], e0, cnt, s);
        float *O = d.O[p];
        if (O == nullptr) return;
        float z[4] = {0.f, 0.f, 0.f, 0.f};
        float sc;
        bool noise;
        noise_scale(f, sc, noise);
        if (noise) {
            const uint64_t st = f.step + (f.step_dev ? *f.step_dev : 0ull);
            uint32_t w[4];
            normals4(q, d.pidx[p], (uint32_t)st, (uint32_t)(st >> 32), f.k0, f.k1, z, w);
        }
        if (cnt == 4 && (d.flags[p] & 2u)) {
            float4 o;
            o.x = (s[0] + sc * z[0]) / f.denom;
            o.y = (s[1] + sc * z[1]) / f.denom;
            o.z = (s[2] + sc * z[2]) / f.denom;
            o.w = (s[3] + sc * z[3]) / f.denom;
            reinterpret_cast<float4 *>(O)[q] = o;
        } else {
            for (int i = 0; i < cnt; ++i) O[e0 + i] = (s[i] + sc * z[i]) / f.denom;
        }
        return;
    }

    const int b = (int)blockIdx.x;
    const int p = find_param(f.cblk0, d.count, b);
    const float *G = d.G[p];
    const i64 numel = d.numel[p];
    const bool vec = (d.flags[p] & 1u) != 0;
    const int grp = tid / kCols, col = tid % kCols;
    // this thread's column: float4 column q (elements 4q..4q+3) or element q
    const i64 q = (i64)(b - f.cblk0[p]) * kCols + col;
    const bool active = vec ? 4 * q < numel : q < numel;
    const i64 N = d.N;
    i64 na = N;
    if (f.n_active) {
        const int64_t v = *f.n_active;
        na = v < 0 ? 0 : (v < N ? v : N);
    }
    const i64 per = ceil_div(N, KG);
    const i64 lo = grp * per < N ? grp * per : N, hi = lo + per < N ? lo + per : N;
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    const float4 *g4 = reinterpret_cast<const float4 *>(G);
    const i64 st4 = numel / 4;

    for (i64 c0 = 0; c0 < N; c0 += kCfChunk) {
        const i64 c1 = c0 + kCfChunk < N ? c0 + kCfChunk : N;
        __syncthreads();   // the previous chunk's factors have been used
        for (i64 n = c0 + tid; n < c1; n += kThreads) {
            float nr;
            if (f.sqnorm) {
                float sq = 0.0f;
                for (int l = 0; l < f.L; ++l) sq += f.sqnorm[(i64)l * N + n];
                nr = n < na ? sqrtf(sq) : -1.0f;
                if (b == 0) {
                    if (!isfinite(nr)) raise_flag(f.status, DP_FLAG_NONFINITE);
                    f.norm[n] = nr;
                }
            } else {
                nr = f.norm[n];
            }
            cfs[n - c0] = clip_factor(nr, f.C);
        }
        __syncthreads();
        const i64 e1 = hi < na ? hi : na;
        const i64 a0 = lo > c0 ? lo : c0, a1 = e1 < c1 ? e1 : c1;
        if (!active || a0 >= a1) continue;
        if (vec) {
            i64 n = a0;
            // eight samples' loads in flight before the (in-order) accumulation
            for (; n + 8 <= a1; n += 8) {
                float4 a[8];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    a[j] = STREAM ? load_stream4(reinterpret_cast<const float *>(g4 + (n + j) * st4 + q))
                                  : g4[(n + j) * st4 + q];
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const float cn = cfs[n + j - c0];
                    acc[0] += cn * a[j].x; acc[1] += cn * a[j].y; acc[2] += cn * a[j].z; acc[3] += cn * a[j].w;
                }
            }
            for (; n < a1; ++n) {
                const float4 a = g4[n * st4 + q];
                const float cn = cfs[n - c0];
                acc[0] += cn * a.x; acc[1] += cn * a.y; acc[2] += cn * a.z; acc[3] += cn * a.w;
            }
        } else {
            i64 n = a0;
            for (; n + 8 <= a1; n += 8) {
                float a[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) a[j] = G[(n + j) * numel + q];
#pragma unroll
                for (int j = 0; j < 8; ++j) acc[0] += cfs[n + j - c0] * a[j];
            }
            for (; n < a1; ++n) acc[0] += cfs[n - c0] * G[n * numel + q];
        }
    }
    // the sample groups' sums, added in group order
    part[grp][col] = make_float4(acc[0], acc[1], acc[2], acc[3]);
    __syncthreads();
    if (grp != 0 || !active) return;
    float s[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < KG; ++k) {
        const float4 v = part[k][col];
        s[0] += v.x; s[1] += v.y; s[2] += v.z; s[3] += v.w;
    }
    // store the clipped sum and the noised average
    const i64 e0 = vec ? 4 * q : q;
    const int cnt = vec ? 4 : 1;
    for (int i = 0; i < cnt; ++i) d.S[p][e0 + i] = s[i];
    accumulate(d.Acc[p], e0, cnt, s);
    float *O = d.O[p];
    if (O == nullptr) return;
    float z[4] = {0.f, 0.f, 0.f, 0.f};
    float sc;
    bool noise;
    noise_scale(f, sc, noise);
    if (noise) {
        const uint64_t st = f.step + (f.step_dev ? *f.step_dev : 0ull);
        uint32_t w[4];
        normals4(e0 >> 2, d.pidx[p], (uint32_t)st, (uint32_t)(st >> 32), f.k0, f.k1, z, w);
    }
    if (vec) {
        for (int i = 0; i < 4; ++i) O[e0 + i] = (s[i] + sc * z[i]) / f.denom;
    } else {
        O[e0] = (s[0] + sc * z[e0 & 3]) / f.denom;
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
        d.Acc[i] = q.accum;
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
        if ((q.numel & 3) == 0 && aligned(q.sum, 16)) f |= 4u;
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

extern "C" size_t dp_norms_clip_noise_workspace_bytes(const dp_param *params, int32_t count, int64_t N)
{
    (void)params;
    (void)count;
    (void)N;
    return 0;
}

static dp_status norms_clip_noise(const float *sqnorm, int32_t n_layers, const dp_param *params, int32_t count,
                                  int64_t N, float *norm, float C, uint64_t seed, uint64_t step,
                                  const uint64_t *step_dev, float sigma, const float *sigma_table,
                                  int64_t table_len, const int64_t *n_active, float denom, int32_t *status,
                                  hipStream_t stream)
{
    DPG_REQUIRE(count >= 0 && N >= 0, DP_EINVAL);
    DPG_REQUIRE(count == 0 || params != nullptr, DP_EINVAL);
    DPG_REQUIRE(C > 0.0f && sigma >= 0.0f && denom > 0.0f, DP_EINVAL);
    DPG_REQUIRE(!(sigma > 0.0f && __builtin_isinf(C)), DP_EINVAL);
    // a schedule may hold positive entries: it needs a finite clipping bound
    DPG_REQUIRE(sigma_table == nullptr || (table_len >= 1 && !__builtin_isinf(C)), DP_EINVAL);
    DPG_REQUIRE(sqnorm == nullptr || n_layers >= 1, DP_EINVAL);
    DPG_REQUIRE(N == 0 || norm != nullptr, DP_EINVAL);
    for (int i = 0; i < count; ++i) {
        const dp_param &q = params[i];
        DPG_REQUIRE(q.numel >= 0 && (q.flags & ~(uint32_t)DP_PARAM_REDUCE) == 0, DP_EINVAL);
        DPG_REQUIRE(q.numel / 4 < (i64(1) << 32), DP_EINVAL);
        DPG_REQUIRE(q.numel == 0 || q.sum != nullptr, DP_EINVAL);
        if (q.flags & DP_PARAM_REDUCE) DPG_REQUIRE(N == 0 || q.numel == 0 || q.grad_sample != nullptr, DP_EINVAL);
    }
    const bool noise = sigma > 0.0f;
    FusedArgs f;
    f.L = n_layers;
    f.norm = norm;
    f.C = C;
    f.k0 = (uint32_t)seed;
    f.k1 = (uint32_t)(seed >> 32);
    f.step = step;
    f.step_dev = step_dev;
    f.sc = noise ? sigma * C : 0.0f;
    f.denom = denom;
    f.noise = noise ? 1 : 0;
    f.sigma_tab = sigma_table;
    f.tab_len = table_len;
    f.n_active = n_active;
    f.status = status;
    bool norms_done = sqnorm == nullptr || N == 0;
    for (int first = 0; first < count; first += kMaxGroup) {
        const int c = count - first < kMaxGroup ? count - first : kMaxGroup;
        GroupDesc d;
        describe(params, first, c, N, d);
        int ob = 0;
        i64 col_bytes = 0;     // per-sample gradient bytes the column reduce reads
        i64 cols[kMaxGroup];   // columns (float4 or single) of each column-reduced tensor, else 0
        for (int i = 0; i < c; ++i) {
            f.oblk0[i] = ob;
            cols[i] = 0;
            const bool col = d.R[i] && N > 0 && d.numel[i] > 0;
            if (col) {
                col_bytes += 4 * N * d.numel[i];
                // 16-byte columns need a 16-byte aligned tensor (the partial flag bit 0
                // of describe() also asks for an aligned sum, which this path does not)
                const bool v = (d.numel[i] & 3) == 0 && aligned(d.G[i], 16);
                d.flags[i] = (d.flags[i] & ~1u) | (v ? 1u : 0u);
                cols[i] = v ? d.numel[i] / 4 : d.numel[i];
            } else {
                ob += (int)ceil_div(ceil_div(d.numel[i], 4), kThreads);
            }
        }
        auto col_blocks = [&](int kg) {
            i64 n = 0;
            for (int i = 0; i < c; ++i) n += ceil_div(cols[i], kThreads / kg);
            return n;
        };
        const int kg = col_blocks(4) >= kMinColBlocks ? 4 : (col_blocks(8) >= kMinColBlocks ? 8 : 16);
        int cb = 0;
        for (int i = 0; i < c; ++i) {
            f.cblk0[i] = cb;
            cb += (int)ceil_div(cols[i], kThreads / kg);
        }
        f.cblk0[c] = cb;
        f.oblk0[c] = ob;
        f.cblocks = cb;
        if (!norms_done && cb == 0) {
            // no column work to compute the norms in: compute them first
            const dp_status st = dp_per_sample_norms_active(sqnorm, n_layers, N, n_active, norm, status, stream);
            if (st != DP_OK) return st;
            norms_done = true;
        }
        f.sqnorm = norms_done ? nullptr : sqnorm;
        if (cb + ob > 0) {
            // stream the gradients when there are many of them (16 MB or more)
            const unsigned grid = (unsigned)(cb + ob);
            const bool stream_loads = col_bytes >= (i64(16) << 20);
            if (kg == 4) {
                if (stream_loads) norms_clip_noise_kernel<true, 4><<<grid, kThreads, 0, stream>>>(d, f);
                else norms_clip_noise_kernel<false, 4><<<grid, kThreads, 0, stream>>>(d, f);
            } else if (kg == 8) {
                if (stream_loads) norms_clip_noise_kernel<true, 8><<<grid, kThreads, 0, stream>>>(d, f);
                else norms_clip_noise_kernel<false, 8><<<grid, kThreads, 0, stream>>>(d, f);
            } else {
                if (stream_loads) norms_clip_noise_kernel<true, 16><<<grid, kThreads, 0, stream>>>(d, f);
                else norms_clip_noise_kernel<false, 16><<<grid, kThreads, 0, stream>>>(d, f);
            }
        }
        norms_done = true;
    }
    return launch_status();
}

extern "C" dp_status dp_norms_clip_noise(const float *sqnorm, int32_t n_layers, const dp_param *params,
                                         int32_t count, int64_t N, float *norm, float C, uint64_t seed,
                                         uint64_t step, const uint64_t *step_dev, float sigma, float denom,
                                         int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)ws;
    (void)ws_bytes;
    return norms_clip_noise(sqnorm, n_layers, params, count, N, norm, C, seed, step, step_dev, sigma, nullptr, 0,
                            nullptr, denom, status, stream);
}

extern "C" dp_status dp_norms_clip_noise_sched(const float *sqnorm, int32_t n_layers, const dp_param *params,
                                               int32_t count, int64_t N, float *norm, float C, uint64_t seed,
                                               uint64_t step, const uint64_t *step_dev, const float *sigma_table,
                                               int64_t table_len, const int64_t *n_active, float denom,
                                               int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)ws;
    (void)ws_bytes;
    DPG_REQUIRE(sigma_table != nullptr, DP_EINVAL);
    return norms_clip_noise(sqnorm, n_layers, params, count, N, norm, C, seed, step, step_dev, 0.0f, sigma_table,
                            table_len, n_active, denom, status, stream);
}

extern "C" dp_status dp_step_advance(uint64_t *step_dev, uint64_t by, hipStream_t stream)
{
    DPG_REQUIRE(step_dev != nullptr, DP_EINVAL);
    step_advance_kernel<<<1, 64, 0, stream>>>(step_dev, by);
    return launch_status();
}
