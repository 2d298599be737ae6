// Conv2d per-sample gradients by implicit im2col on MFMA.
//
// For sample n the weight gradient is the product of the output backprop
// GY_n [Cout][L] (L = Ho*Wo positions) with the transposed unfold of the
// input, U_n [L][Cin*kh*kw], whose column (ci, u, v) at position (oh, ow)
// is X_n[ci][oh*sh+u-ph][ow*sw+v-pw] (zero in the padding).  The unfold is
// never written to memory: each K-chunk of positions gathers its slice of
// U_n straight into LDS.  M = Cout, N = Cin*kh*kw, K = L.
#include "common.hpp"
#include "mfma_tile.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 64, kBN = 64, kBK = 32;

struct ConvShape {
    i64 Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
};

template <typename T>
__global__ __launch_bounds__(kThreads) void conv_per_sample_kernel(
    const T *__restrict__ X, const T *__restrict__ GY, ConvShape s, int tiles_n, int tiles,
    float scale, float *__restrict__ gW, float *__restrict__ gb, float *__restrict__ partial)
{
    __shared__ float As[kBK * kBM];
    __shared__ float Bs[kBK * kBN];
    __shared__ float red[16];
    const i64 n = blockIdx.x / tiles;
    const int tile = blockIdx.x % tiles;
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const i64 m0 = (i64)tm * kBM, n0 = (i64)tn * kBN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * (kBM / 2), wn = (wave & 1) * (kBN / 2);
    const i64 L = s.Ho * s.Wo;
    const i64 KK = s.Cin * s.kh * s.kw;
    const i64 khw = s.kh * s.kw;
    const T *Xn = X + n * s.Cin * s.H * s.W;
    const T *Gn = GY + n * s.Cout * L;
    const bool do_bias = gb != nullptr && tn == 0;

    MfmaTile<kBM, kBN> t;
    t.zero();
    float bias_acc = 0.0f;

    for (i64 k0 = 0; k0 < L; k0 += kBK) {
        // A operand: As[kk][ii] = GY_n[m0+ii][k0+kk] (consecutive threads walk positions)
        for (int e = tid; e < kBK * kBM; e += kThreads) {
            const int ii = e / kBK, kk = e % kBK;
            const i64 p = k0 + kk, co = m0 + ii;
            As[kk * kBM + ii] = (p < L && co < s.Cout) ? load_elem<T>(Gn, co * L + p) : 0.0f;
        }
        // B operand: Bs[kk][jj] = U_n[k0+kk][n0+jj], gathered from the input
        for (int e = tid; e < kBK * kBN; e += kThreads) {
            const int jj = e / kBK, kk = e % kBK;
            const i64 p = k0 + kk, j = n0 + jj;
            float v = 0.0f;
            if (p < L && j < KK) {
                const i64 ci = j / khw, rem = j % khw;
                const i64 u = rem / s.kw, vv = rem % s.kw;
                const i64 oh = p / s.Wo, ow = p % s.Wo;
                const i64 ih = oh * s.sh + u - s.ph, iw = ow * s.sw + vv - s.pw;
                if (ih >= 0 && ih < s.H && iw >= 0 && iw < s.W)
                    v = load_elem<T>(Xn, (ci * s.H + ih) * s.W + iw);
            }
            Bs[kk * kBN + jj] = v;
        }
        __syncthreads();
        t.template mma<kBK>(As, kBM, Bs, kBN, wm, wn, lane);
        if (do_bias && tid < kBM) {
#pragma unroll 8
            for (int kk = 0; kk < kBK; ++kk) bias_acc += As[kk * kBM + tid];
        }
        __syncthreads();
    }

    float sq = 0.0f;
    float *G = gW + n * s.Cout * KK;
    t.for_each(wm, wn, lane, [&](int r, int c, float v) {
        const i64 i = m0 + r, j = n0 + c;
        if (i < s.Cout && j < KK) {
            const float g = scale * v;
            G[i * KK + j] = g;
            sq += g * g;
        }
    });
    if (do_bias && tid < kBM && m0 + tid < s.Cout) {
        const float g = scale * bias_acc;
        gb[n * s.Cout + m0 + tid] = g;
        sq += g * g;
    }
    sq = block_sum(sq, red);
    if (partial && tid == 0) partial[n * tiles + tile] = sq;
}

__global__ void conv_reduce_partials_kernel(const float *__restrict__ partial, i64 N, int tiles,
                                            float *__restrict__ sqnorm)
{
    const i64 n = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (n >= N) return;
    float s = 0.0f;
    for (int t = 0; t < tiles; ++t) s += partial[n * tiles + t];
    sqnorm[n] = s;
}

int conv_tiles(i64 Cin, i64 Cout, i64 kh, i64 kw, int *tiles_n)
{
    *tiles_n = (int)ceil_div(Cin * kh * kw, kBN);
    return (int)ceil_div(Cout, kBM) * *tiles_n;
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_grad_sample_conv2d_workspace_bytes(int64_t N, int64_t Cin, int64_t Cout,
                                                        int64_t kh, int64_t kw)
{
    if (N <= 0 || Cin <= 0 || Cout <= 0 || kh <= 0 || kw <= 0) return 0;
    int tn;
    const int tiles = conv_tiles(Cin, Cout, kh, kw, &tn);
    return (size_t)(N * tiles) * sizeof(float);
}

extern "C" dp_status dp_grad_sample_conv2d(const void *X, const void *GY, dp_dtype dt, int64_t N,
                                           int64_t Cin, int64_t H, int64_t W, int64_t Cout,
                                           int64_t Ho, int64_t Wo, int64_t kh, int64_t kw,
                                           int64_t sh, int64_t sw, int64_t ph, int64_t pw,
                                           int64_t dh, int64_t dw, int64_t groups, float scale,
                                           float *gW, float *gb, float *sqnorm, int32_t *status,
                                           void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && Cin >= 1 && H >= 1 && W >= 1 && Cout >= 1, DP_EINVAL);
    DPG_REQUIRE(kh >= 1 && kw >= 1 && sh >= 1 && sw >= 1 && ph >= 0 && pw >= 0, DP_EINVAL);
    DPG_REQUIRE(groups >= 1 && dh >= 1 && dw >= 1, DP_EINVAL);
    DPG_REQUIRE(groups == 1 && dh == 1 && dw == 1, DP_EUNSUPPORTED);
    DPG_REQUIRE(H + 2 * ph >= kh && W + 2 * pw >= kw, DP_EINVAL);
    DPG_REQUIRE(Ho == (H + 2 * ph - kh) / sh + 1 && Wo == (W + 2 * pw - kw) / sw + 1, DP_EINVAL);
    DPG_REQUIRE(N == 0 || (X != nullptr && GY != nullptr && gW != nullptr), DP_EINVAL);
    const size_t need = dp_grad_sample_conv2d_workspace_bytes(N, Cin, Cout, kh, kw);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;

    ConvShape s{Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw};
    int tiles_n;
    const int tiles = conv_tiles(Cin, Cout, kh, kw, &tiles_n);
    float *partial = sqnorm ? (float *)ws : nullptr;
    const dim3 grid((unsigned)(N * tiles));
    if (dt == DP_F32)
        conv_per_sample_kernel<float><<<grid, kThreads, 0, stream>>>(
            (const float *)X, (const float *)GY, s, tiles_n, tiles, scale, gW, gb, partial);
    else
        conv_per_sample_kernel<uint16_t><<<grid, kThreads, 0, stream>>>(
            (const uint16_t *)X, (const uint16_t *)GY, s, tiles_n, tiles, scale, gW, gb, partial);
    if (sqnorm)
        conv_reduce_partials_kernel<<<(unsigned)ceil_div(N, 256), 256, 0, stream>>>(partial, N, tiles,
                                                                                   sqnorm);
    return launch_status();
}
