// Ghost norms: the per-sample gradient norm of a Linear layer over a sequence
// without forming the per-sample gradient.
//
// The paper's related-work section ("Gradient Clipping") contrasts Opacus'
// materialized per-sample gradients with methods that compute only each
// sample's gradient norm (exactly, for fully connected layers), and names
// their extension to sequential inputs ("ghost clipping") as the improvement
// Opacus plans to take up.  For gW_n = s * B_n^T A_n (d_out x d_in, summed
// over T positions) and gb_n = s * sum_t B_n,t:
//
//   |gW_n|^2 = s^2 <A_n A_n^T, B_n B_n^T>_F,     |gb_n|^2 = s^2 1^T (B_n B_n^T) 1,
//
// so sqnorm_n = s^2 * sum_{t,t'} G_B[t][t'] * (G_A[t][t'] + bias), with the
// T x T Gram matrices G_A = A_n A_n^T and G_B = B_n B_n^T.  That costs
// 2 T^2 (d_in + d_out) flops per sample against 2 T d_in d_out for the
// gradient, and writes one float per sample instead of d_out * d_in.
//
// Kernels.  (1) `ghost_gram_kernel`: one workgroup per (sample, 64 x 64
// tile pair (bi <= bj) of the Gram matrices, chunk of features of A or of
// B); it writes that chunk's contribution to the tile of G_A or G_B.  Both
// Grams contract over the feature index, which is the contiguous one in
// memory, so each MFMA operand is eight (bf16) or one (fp32) consecutive
// features of one position row: stages of 32 features of the tile's 2 x 64
// rows are copied to LDS with 16-byte loads (double buffered, the next
// stage's loads in flight during the current stage's MFMAs) and read back
// with one ds_read per operand.  Wave w computes the 32 x 32 sub-tile
// (w & 1, w >> 1); rows past T are staged as zeros.  The feature chunks
// exist to give a small batch enough workgroups to fill the GPU.  (2)
// `ghost_combine_kernel`: per (sample, tile pair), adds the chunks of G_A and
// of G_B in chunk order (the tiles share one register layout, so this is
// elementwise), forms sum G_B (G_A + bias), counts off-diagonal pairs twice
// (the Grams are symmetric) and writes s^2 times that; the pairs of a sample
// are then added in pair order.
#include "common.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kBT = 64;            // Gram tile edge (positions)
constexpr int kKC = 32;            // features per stage
constexpr int kRows = 2 * kBT;     // staged rows: the tile's i-block, then its j-block

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <typename T>
struct Elem;

template <>
struct Elem<uint16_t> {
    static constexpr int ROW = 80;            // 64 bytes of features + 16 of padding (spreads the banks)
};

template <>
struct Elem<float> {
    static constexpr int ROW = 144;           // 128 + 16
};

template <typename T>
constexpr int kChunks = (kRows * kKC * (int)sizeof(T)) / 16 / kThreads;   // 16-byte chunks per thread per stage

constexpr int kPerChunk(int elem_bytes) { return 16 / elem_bytes; }

// (bi, bj), bi <= bj, of pair p in row-major order of the upper triangle
__device__ __forceinline__ void pair_of(int p, int nb, int &bi, int &bj)
{
    bi = 0;
    while (p >= nb - bi) {
        p -= nb - bi;
        ++bi;
    }
    bj = bi + p;
}

// One stage's loads for this thread: chunk q = tid + kThreads * c covers
// staged row q / CPR, features (q % CPR) * PC .. + PC - 1 of rows of length
// ld; features at or past fend read as zeros.
template <typename T, bool VEC>
struct StageRegs {
    uint4 v[kChunks<T>];
};

template <typename T, bool VEC>
__device__ __forceinline__ void load_stage(const T *X, i64 Tn, i64 ld, i64 fend, int bi, int bj, i64 f0, int tid,
                                           StageRegs<T, VEC> &r)
{
    constexpr int PC = kPerChunk(sizeof(T));
    constexpr int CPR = kKC / PC;
#pragma unroll
    for (int c = 0; c < kChunks<T>; ++c) {
        const int q = tid + kThreads * c;
        const int row = q / CPR, cc = q % CPR;
        const i64 t = row < kBT ? (i64)bi * kBT + row : (i64)bj * kBT + (row - kBT);
        const i64 f = f0 + (i64)cc * PC;
        if (VEC) {
            uint4 z = make_uint4(0u, 0u, 0u, 0u);
            if (t < Tn && f < fend) z = *reinterpret_cast<const uint4 *>(X + t * ld + f);
            r.v[c] = z;
        } else {
            T e[PC];
#pragma unroll
            for (int k = 0; k < PC; ++k) e[k] = (t < Tn && f + k < fend) ? X[t * ld + f + k] : T(0);
            r.v[c] = *reinterpret_cast<const uint4 *>(e);
        }
    }
}

template <typename T, bool VEC>
__device__ __forceinline__ void store_stage(char *L, int tid, const StageRegs<T, VEC> &r)
{
    constexpr int CPR = kKC / kPerChunk(sizeof(T));
#pragma unroll
    for (int c = 0; c < kChunks<T>; ++c) {
        const int q = tid + kThreads * c;
        const int row = q / CPR, cc = q % CPR;
        *reinterpret_cast<uint4 *>(L + row * Elem<T>::ROW + cc * 16) = r.v[c];
    }
}

// The stage's MFMAs for the wave's sub-tile: rows ra (i side) and rb (j side)
// of the staged tile are this lane's operand rows.
__device__ __forceinline__ void mma_stage(const char *L, int ra, int rb, int lane, f32x16_t &acc, uint16_t)
{
    constexpr int ROW = Elem<uint16_t>::ROW;
#pragma unroll
    for (int ks = 0; ks < kKC / 16; ++ks) {
        const int off = ks * 32 + 16 * (lane >> 5);
        const bf16x8_t a = *reinterpret_cast<const bf16x8_t *>(L + ra * ROW + off);
        const bf16x8_t b = *reinterpret_cast<const bf16x8_t *>(L + rb * ROW + off);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc, 0, 0, 0);
    }
}

__device__ __forceinline__ void mma_stage(const char *L, int ra, int rb, int lane, f32x16_t &acc, float)
{
    constexpr int ROW = Elem<float>::ROW;
#pragma unroll
    for (int ks = 0; ks < kKC / 2; ++ks) {
        const int off = 4 * (2 * ks + (lane >> 5));
        const float a = *reinterpret_cast<const float *>(L + ra * ROW + off);
        const float b = *reinterpret_cast<const float *>(L + rb * ROW + off);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
    }
}

template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void ghost_gram_kernel(const T *__restrict__ A, const T *__restrict__ B,
                                                              i64 Tn, i64 din, i64 dout, int nb, int pairs, int kch,
                                                              int ca, int chunks, float *__restrict__ tiles)
{
    __shared__ __attribute__((aligned(16))) char lds[2][kRows * Elem<T>::ROW];
    const int c = (int)(blockIdx.x % chunks);
    const i64 np = blockIdx.x / chunks;
    const i64 n = np / pairs;
    const int p = (int)(np % pairs);
    int bi, bj;
    pair_of(p, nb, bi, bj);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int ra = 32 * (wave & 1) + (lane & 31);          // i-side row of the lane's operand
    const int rb = kBT + 32 * (wave >> 1) + (lane & 31);   // j-side row
    const bool onA = c < ca;
    const i64 d = onA ? din : dout;
    const T *X = onA ? A + n * Tn * din : B + n * Tn * dout;
    const i64 f_begin = (i64)(onA ? c : c - ca) * kch;
    const i64 f_end = f_begin + kch < d ? f_begin + kch : d;
    const int stages = (int)ceil_div(f_end - f_begin, kKC);

    f32x16_t acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.0f;

    StageRegs<T, VEC> regs;
    load_stage<T, VEC>(X, Tn, d, f_end, bi, bj, f_begin, tid, regs);
    store_stage<T, VEC>(lds[0], tid, regs);
    __syncthreads();
    for (int st = 0; st < stages; ++st) {
        const bool more = st + 1 < stages;
        if (more) load_stage<T, VEC>(X, Tn, d, f_end, bi, bj, f_begin + (i64)(st + 1) * kKC, tid, regs);
        mma_stage(lds[st & 1], ra, rb, lane, acc, T());
        if (more) store_stage<T, VEC>(lds[(st + 1) & 1], tid, regs);
        __syncthreads();
    }
    // the tile in register order: wave, lane, register
    float4 *o = reinterpret_cast<float4 *>(tiles + (size_t)blockIdx.x * (kBT * kBT) + wave * 1024 + lane * 16);
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
}

// one workgroup per (sample, pair); thread i owns entries 16 i .. 16 i + 15
__global__ __launch_bounds__(kThreads) void ghost_combine_kernel(const float *__restrict__ tiles, int nb, int pairs,
                                                                 int ca, int chunks, float bias, float s2,
                                                                 float *__restrict__ out)
{
    __shared__ float red[kThreads / kWave];
    const int p = (int)(blockIdx.x % pairs);
    int bi, bj;
    pair_of(p, nb, bi, bj);
    const float *base = tiles + (size_t)blockIdx.x * chunks * (kBT * kBT) + threadIdx.x * 16;
    float ga[16], gb[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) ga[r] = gb[r] = 0.0f;
    for (int c = 0; c < chunks; ++c) {
        const float4 *t = reinterpret_cast<const float4 *>(base + (size_t)c * (kBT * kBT));
        float v[16];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 x = t[q];
            v[4 * q] = x.x; v[4 * q + 1] = x.y; v[4 * q + 2] = x.z; v[4 * q + 3] = x.w;
        }
        if (c < ca) {
#pragma unroll
            for (int r = 0; r < 16; ++r) ga[r] += v[r];
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r) gb[r] += v[r];
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += gb[r] * (ga[r] + bias);
    s = wave_sum(s);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kThreads / kWave; ++w) t += red[w];
        out[blockIdx.x] = s2 * (bi == bj ? t : 2.0f * t);
    }
}

int tile_pairs(i64 T)
{
    const i64 nb = ceil_div(T, kBT);
    return (int)(nb * (nb + 1) / 2);
}

// feature chunk per workgroup: enough (sample, pair, chunk) workgroups to
// give every CU a few, in whole stages
struct GhostPlan {
    int nb, pairs, kch, ca, cb, chunks;
};

GhostPlan ghost_plan(i64 N, i64 Tn, i64 din, i64 dout)
{
    GhostPlan g;
    g.nb = (int)ceil_div(Tn, kBT);
    g.pairs = tile_pairs(Tn);
    const i64 want = ceil_div(1024, N * g.pairs > 0 ? N * g.pairs : 1);       // chunks per (sample, pair)
    i64 kch = ceil_div(din + dout, want);
    kch = ceil_div(kch, kKC) * kKC;
    if (kch < 256) kch = 256;
    g.kch = (int)kch;
    g.ca = (int)ceil_div(din, kch);
    g.cb = (int)ceil_div(dout, kch);
    g.chunks = g.ca + g.cb;
    return g;
}

template <typename T>
void launch_ghost(const void *A, const void *B, i64 N, i64 Tn, i64 din, i64 dout, bool vec, const GhostPlan &g,
                  float *tiles, hipStream_t stream)
{
    const dim3 grid((unsigned)(N * g.pairs * g.chunks));
    if (vec)
        ghost_gram_kernel<T, true><<<grid, kThreads, 0, stream>>>((const T *)A, (const T *)B, Tn, din, dout, g.nb,
                                                                  g.pairs, g.kch, g.ca, g.chunks, tiles);
    else
        ghost_gram_kernel<T, false><<<grid, kThreads, 0, stream>>>((const T *)A, (const T *)B, Tn, din, dout, g.nb,
                                                                   g.pairs, g.kch, g.ca, g.chunks, tiles);
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_ghost_norm_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in, int64_t d_out)
{
    if (N <= 0 || T <= 0 || d_in <= 0 || d_out <= 0) return 0;
    const GhostPlan g = ghost_plan(N, T, d_in, d_out);
    // the chunks' Gram tiles, then (several pairs) one partial per (sample, pair)
    size_t b = (size_t)(N * g.pairs * g.chunks) * (kBT * kBT) * sizeof(float);
    if (g.pairs > 1) b += (size_t)(N * g.pairs) * sizeof(float);
    return b;
}

extern "C" dp_status dp_ghost_norm_linear(const void *A, const void *B, dp_dtype dt, int64_t N, int64_t T,
                                          int64_t d_in, int64_t d_out, float scale, int32_t bias, float *sqnorm,
                                          int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && T >= 0 && d_in >= 1 && d_out >= 1, DP_EINVAL);
    DPG_REQUIRE(N < (i64(1) << 31) && T < (i64(1) << 20) && d_in < (i64(1) << 31) && d_out < (i64(1) << 31),
                DP_EINVAL);
    DPG_REQUIRE(N == 0 || sqnorm != nullptr, DP_EINVAL);
    DPG_REQUIRE(N * T == 0 || (A != nullptr && B != nullptr), DP_EINVAL);
    if (N > 0 && T > 0) {
        const GhostPlan g = ghost_plan(N, T, d_in, d_out);
        DPG_REQUIRE(N * g.pairs * g.chunks < (i64(1) << 31), DP_EUNSUPPORTED);
    }
    const size_t need = dp_ghost_norm_linear_workspace_bytes(N, T, d_in, d_out);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;
    if (T == 0) {
        zero_fill(sqnorm, N, stream);
        return launch_status();
    }
    const GhostPlan g = ghost_plan(N, T, d_in, d_out);
    const i64 pc = 16 / (i64)dtype_bytes(dt);
    const bool vec = d_in % pc == 0 && d_out % pc == 0 && aligned(A, 16) && aligned(B, 16);
    float *tiles = (float *)ws;
    float *part = tiles + (size_t)(N * g.pairs * g.chunks) * (kBT * kBT);
    if (dt == DP_BF16) launch_ghost<uint16_t>(A, B, N, T, d_in, d_out, vec, g, tiles, stream);
    else launch_ghost<float>(A, B, N, T, d_in, d_out, vec, g, tiles, stream);
    float *out = g.pairs > 1 ? part : sqnorm;
    ghost_combine_kernel<<<(unsigned)(N * g.pairs), kThreads, 0, stream>>>(tiles, g.nb, g.pairs, g.ca, g.chunks,
                                                                          bias ? 1.0f : 0.0f, scale * scale, out);
    if (g.pairs > 1) sum_partials(part, N, g.pairs, sqnorm, stream);
    return launch_status();
}
