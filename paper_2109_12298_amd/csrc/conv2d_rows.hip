// Per-sample Conv2d gradients for samples whose input planes do not fit one
// workgroup's LDS (the CIFAR network's convolutions, for example), by output
// row chunks.
//
// gW_n[co][kk] = s * sum_p GY_n[co][p] * X_n[ci][oh*sh+u-ph][ow*sw+v-pw],
// kk = (ci, u, v), p = (oh, ow)   (the weight gradient of the
// cross-correlation restricted to sample n; zero outside the input).
//
// A workgroup owns one sample's gradient tile of up to 288 weight columns
// (nine MFMA blocks of 32) by 64 (or 32) output channels, with every
// accumulator of the tile in registers, and walks the sample's output rows in
// chunks.  Per chunk it stages the input rows the chunk reads (for the tile's
// input channels, with a zero halo) and the chunk's backprop, then contracts
// over the chunk's positions on v_mfma_f32_32x32x2_f32: per position pair a
// lane reads one unfold element per block (its column's offset plus the
// position's, from a table) and one backprop element, and the same position
// work feeds up to five MFMAs.  Against tiling the unfold by columns and
// staging whole planes, this stages each backprop element once per column
// tile instead of once per 32 columns, and keeps the index arithmetic per
// MFMA small (the tiled kernel was bound by it, not by the matrix unit).
//
// The backprop chunk sits in LDS as [position pair][channel][parity] with a
// pair stride of 2 * channels + 2 floats: the two positions of a pair (the
// two halves of the wave) read different banks, and the staging writes, whose
// consecutive lanes take consecutive pairs of one channel (coalesced loads),
// spread over the banks.
// A sample's norm partials (one per tile) are added in tile order by a
// second kernel; a single tile writes the norm directly.
#include "common.hpp"
#include "conv2d_rows.hpp"

namespace dpg {
namespace {

typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kMaxBlk = 9;                 // 32-column blocks per tile
constexpr int kRowsLds = 60 * 1024;        // dynamic LDS budget (two workgroups per CU)

struct RowsShape {
    int Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
    int Wp, L, KK, khw;
    int nblk;             // 32-column blocks per tile (<= 9)
    int ktiles, ctiles;   // column tiles, channel tiles
    int np;               // input channels a column tile touches (upper bound)
    int RC, XR;           // output rows per chunk, staged input rows per chunk
    int PC;               // positions per chunk, RC * Wo rounded up to even
    int x_floats;         // np * XR * Wp
    int vec;              // float4 stores of gW
    float inv_khw, inv_kw, inv_wo;
    // stepping an element index by kThreads in the input stage [np][XR][Wp]
    // (channel, row, column) and in the backprop stage (channel, pair)
    int xs_c, xs_r, xs_w, gs_c, gs_p;
    float inv_xrw, inv_wp, inv_pairs;
};

__device__ __forceinline__ void fdivmod(int x, int d, float inv_d, int &q, int &r)
{
    q = (int)((float)x * inv_d);
    r = x - q * d;
    q += (r >= d ? 1 : 0) - (r < 0 ? 1 : 0);
    r = x - q * d;
}

// WCO: 32-channel blocks per tile (1 or 2).  The waves form (4 / WCO) column
// rows x WCO channel columns; wave row q takes blocks q, q + 4/WCO, ...
template <typename T, int WCO>
__global__ __launch_bounds__(kThreads, 2) void conv_rows_kernel(const T *__restrict__ X, const T *__restrict__ GY,
                                                                RowsShape s, float scale, float *__restrict__ gW,
                                                                float *__restrict__ gb, float *__restrict__ sqout,
                                                                int direct)
{
    constexpr int WKK = kWaves / WCO;
    constexpr int FM = (kMaxBlk + WKK - 1) / WKK;
    constexpr int BN = 32 * WCO;
    extern __shared__ __attribute__((aligned(16))) float lds[];
    __shared__ float red[kWaves];
    __shared__ float bsum[kThreads];          // bias partials [segment][channel]

    const int tiles = s.ktiles * s.ctiles;
    const i64 n = blockIdx.x / tiles;
    const int tile = (int)(blockIdx.x % tiles);
    const int tk = tile / s.ctiles, tc = tile % s.ctiles;
    const int m0 = tk * s.nblk * 32;          // first weight column
    const int n0 = tc * BN;                   // first output channel
    const int ci0 = m0 / s.khw;
    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wq = wave / WCO, wc = wave % WCO;
    float *Xs = lds;                                   // [np][XR][Wp]
    constexpr int GSP = 2 * BN + 2;                    // floats per position pair
    float *Gs = lds + s.x_floats;                      // [PC/2][BN][2], pair stride GSP
    int *Pt = reinterpret_cast<int *>(Gs + s.PC / 2 * GSP);   // [PC] offset of position p in the staged rows
    const T *Xn = X + n * (i64)s.Cin * s.H * s.W;
    const T *Gn = GY + n * (i64)s.Cout * s.L;
    const int cvalid = s.Cout - n0 < BN ? s.Cout - n0 : BN;

    // the lane's unfold column offsets in the staged rows (a column past the
    // tile or the weight reads offset 0; its output rows are never stored)
    int koff[FM];
    bool bon[FM];
#pragma unroll
    for (int x = 0; x < FM; ++x) {
        const int blk = wq + WKK * x;
        bon[x] = blk < s.nblk;
        const int kk = m0 + blk * 32 + (lane & 31);
        koff[x] = 0;
        if (bon[x] && kk < s.KK) {
            int ci, rem, u, v;
            fdivmod(kk, s.khw, s.inv_khw, ci, rem);
            fdivmod(rem, s.kw, s.inv_kw, u, v);
            koff[x] = (ci - ci0) * s.XR * s.Wp + u * s.Wp + v;
        }
    }
    f32x16_t acc[FM];
#pragma unroll
    for (int x = 0; x < FM; ++x)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[x][r] = 0.0f;
    const bool do_bias = gb != nullptr && tk == 0;
    float bacc = 0.0f;    // bias: thread (bseg, bco) adds positions bseg, bseg + kSegs, ... of each chunk
    const int bco = tid % BN, bseg = tid / BN;
    constexpr int kSegs = kThreads / BN;
    // the thread's first element in each stage
    int xc0, xr0, xw0, gc0, gp0;
    {
        int rem;
        fdivmod(tid, s.XR * s.Wp, s.inv_xrw, xc0, rem);
        fdivmod(rem, s.Wp, s.inv_wp, xr0, xw0);
        fdivmod(tid, s.PC / 2, s.inv_pairs, gc0, gp0);
    }

    for (int oh0 = 0; oh0 < s.Ho; oh0 += s.RC) {
        const int rows = s.Ho - oh0 < s.RC ? s.Ho - oh0 : s.RC;
        const int len = rows * s.Wo;                   // positions of this chunk
        const int pbase = oh0 * s.Wo;
        const int ih0 = oh0 * s.sh - s.ph;
        __syncthreads();                               // the previous chunk is consumed
        // ---- input rows ih0 .. ih0 + XR - 1 of the tile's channels, zero
        // outside.  Thread elements tid, tid + kThreads, ... of [np][XR][Wp];
        // their (channel, row, column) are stepped, not divided out.
        {
            int c = xc0, r = xr0, w = xw0;
            for (int idx = tid; idx < s.np * s.XR * s.Wp; idx += kThreads) {
                const int ci = ci0 + c, ih = ih0 + r, iw = w - s.pw;
                const bool in = ci < s.Cin && ih >= 0 && ih < s.H && iw >= 0 && iw < s.W;
                Xs[idx] = in ? load_elem<T>(Xn, ((i64)ci * s.H + ih) * s.W + iw) : 0.0f;
                w += s.xs_w;
                if (w >= s.Wp) {
                    w -= s.Wp;
                    ++r;
                }
                r += s.xs_r;
                if (r >= s.XR) {
                    r -= s.XR;
                    ++c;
                }
                c += s.xs_c;
            }
        }
        // ---- the chunk's backprop as [pair][channel][parity], zero past len;
        // consecutive threads take consecutive pairs of one channel (coalesced
        // loads), (channel, pair) stepped like the input's indices
        {
            int co = gc0, pr = gp0;
            for (int e = tid; e < BN * (s.PC / 2); e += kThreads) {
                const int p = 2 * pr;
                const bool cin = co < cvalid;
                const T *src = Gn + (i64)(n0 + co) * s.L + pbase;
                const float g0 = cin && p < len ? load_elem<T>(src, p) : 0.0f;
                const float g1 = cin && p + 1 < len ? load_elem<T>(src, p + 1) : 0.0f;
                *reinterpret_cast<float2 *>(Gs + pr * GSP + 2 * co) = make_float2(g0, g1);
                pr += s.gs_p;
                if (pr >= s.PC / 2) {
                    pr -= s.PC / 2;
                    ++co;
                }
                co += s.gs_c;
            }
        }
        for (int p = tid; p < s.PC; p += kThreads) {
            int oh, ow;
            fdivmod(p, s.Wo, s.inv_wo, oh, ow);
            Pt[p] = p < len ? oh * s.sh * s.Wp + ow * s.sw : 0;
        }
        __syncthreads();
        if (do_bias) {
            // thread (bseg, bco): positions bseg, bseg + kSegs, ... of the chunk, in order
            for (int p = bseg; p < len; p += kSegs) bacc += Gs[(p >> 1) * GSP + 2 * bco + (p & 1)];
        }
        // ---- contraction over the chunk's position pairs; the next pair's
        // reads are issued before the current pair's MFMAs
        const int npairs = (len + 1) >> 1;
        const int gl = wc * 32 + (lane & 31);
        // whole pairs two at a time without masks, then what is left masked
        const int qfull = (len >> 2) << 1;
        for (int q = 0; q < qfull; q += 2) {
            float a[2][FM], b[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int pr = q + h;
                const int po = Pt[2 * pr + half];
                b[h] = Gs[pr * GSP + 2 * gl + half];
#pragma unroll
                for (int x = 0; x < FM; ++x) a[h][x] = Xs[koff[x] + po];
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int x = 0; x < FM; ++x)
                    if (bon[x]) acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[h][x], b[h], acc[x], 0, 0, 0);
        }
        for (int q = qfull; q < npairs; q += 2) {
            float a[2][FM], b[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int pr = q + h < npairs ? q + h : npairs - 1;
                const int p = 2 * pr + half;
                const int po = Pt[p];
                // a position past the chunk (the second of a last, odd pair,
                // or a pair past the end) contributes exactly zero
                const bool pin = q + h < npairs && p < len;
                const float bv = Gs[pr * GSP + 2 * gl + half];
                b[h] = pin ? bv : 0.0f;
#pragma unroll
                for (int x = 0; x < FM; ++x) {
                    const float av = Xs[koff[x] + po];
                    a[h][x] = pin ? av : 0.0f;
                }
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int x = 0; x < FM; ++x)
                    if (bon[x]) acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[h][x], b[h], acc[x], 0, 0, 0);
        }
    }

    // ---- store the tile and its squared norm
    float sq = 0.0f;
    const int co = n0 + wc * 32 + (lane & 31);
    float *G = gW + n * (i64)s.Cout * s.KK;
#pragma unroll
    for (int x = 0; x < FM; ++x) {
        if (!bon[x] || co >= s.Cout) continue;
        const int kb = m0 + (wq + WKK * x) * 32;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
            const int kk = kb + 8 * rb + 4 * half;
            const float g0 = scale * acc[x][4 * rb + 0], g1 = scale * acc[x][4 * rb + 1];
            const float g2 = scale * acc[x][4 * rb + 2], g3 = scale * acc[x][4 * rb + 3];
            const int kend = m0 + s.nblk * 32 < s.KK ? m0 + s.nblk * 32 : s.KK;
            float *dst = G + (i64)co * s.KK + kk;
            if (s.vec && kk + 3 < kend) {
                *reinterpret_cast<float4 *>(dst) = make_float4(g0, g1, g2, g3);
                sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
            } else {
                if (kk + 0 < kend) { dst[0] = g0; sq += g0 * g0; }
                if (kk + 1 < kend) { dst[1] = g1; sq += g1 * g1; }
                if (kk + 2 < kend) { dst[2] = g2; sq += g2 * g2; }
                if (kk + 3 < kend) { dst[3] = g3; sq += g3 * g3; }
            }
        }
    }
    if (do_bias) {
        bsum[bseg * BN + bco] = bacc;
        __syncthreads();
        if (tid < BN && n0 + tid < s.Cout) {
            float b = 0.0f;
#pragma unroll
            for (int k = 0; k < kSegs; ++k) b += bsum[k * BN + tid];
            b *= scale;
            gb[n * s.Cout + n0 + tid] = b;
            sq += b * b;
        }
    }
    sq = wave_sum(sq);
    if (lane == 0) red[wave] = sq;
    __syncthreads();
    if (tid == 0 && sqout) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += red[w];
        if (direct) sqout[n] = t;
        else sqout[n * tiles + tile] = t;
    }
}

bool plan_rows(const ConvRowsArgs &a, RowsShape &s)
{
    s.Cin = (int)a.Cin; s.H = (int)a.H; s.W = (int)a.W; s.Cout = (int)a.Cout;
    s.Ho = (int)a.Ho; s.Wo = (int)a.Wo;
    s.kh = (int)a.kh; s.kw = (int)a.kw; s.sh = (int)a.sh; s.sw = (int)a.sw; s.ph = (int)a.ph; s.pw = (int)a.pw;
    s.Wp = s.W + 2 * s.pw;
    s.L = s.Ho * s.Wo;
    s.khw = s.kh * s.kw;
    s.KK = s.Cin * s.khw;
    const int blocks = (s.KK + 31) / 32;
    s.ktiles = (blocks + kMaxBlk - 1) / kMaxBlk;
    s.nblk = (blocks + s.ktiles - 1) / s.ktiles;          // balanced column tiles
    const int wco = s.Cout > 32 ? 2 : 1;
    s.ctiles = (s.Cout + 32 * wco - 1) / (32 * wco);
    s.np = (s.nblk * 32 + s.khw - 1) / s.khw + 1;
    if (s.np > s.Cin) s.np = s.Cin;
    // the largest row chunk whose stage fits: np * XR * Wp + PC * BN + PC
    const int BN = 32 * wco;
    s.RC = 0;
    for (int rc = s.Ho; rc >= 1; --rc) {
        const int xr = (rc - 1) * s.sh + s.kh;
        const int pc = (rc * s.Wo + 1) & ~1;
        const long fl = (long)s.np * xr * s.Wp + 3 + (long)pc / 2 * (2 * BN + 2) + pc;
        if (fl * 4 <= kRowsLds) {
            s.RC = rc;
            break;
        }
    }
    if (s.RC == 0) return false;
    s.XR = (s.RC - 1) * s.sh + s.kh;
    s.PC = (s.RC * s.Wo + 1) & ~1;
    s.x_floats = s.np * s.XR * s.Wp;
    s.x_floats = (s.x_floats + 3) & ~3;       // keeps the backprop's float2 stores 8-byte aligned
    s.vec = 0;
    s.inv_khw = 1.0f / (float)s.khw;
    s.inv_kw = 1.0f / (float)s.kw;
    s.inv_wo = 1.0f / (float)s.Wo;
    s.inv_xrw = 1.0f / (float)(s.XR * s.Wp);
    s.inv_wp = 1.0f / (float)s.Wp;
    s.inv_pairs = 1.0f / (float)(s.PC / 2);
    {
        const int rows = kThreads / s.Wp;
        s.xs_w = kThreads % s.Wp;
        s.xs_r = rows % s.XR;
        s.xs_c = rows / s.XR;
        s.gs_p = kThreads % (s.PC / 2);
        s.gs_c = kThreads / (s.PC / 2);
    }
    // index arithmetic through float reciprocals needs values below 2^22
    return (long)s.x_floats < (1L << 22) && (long)s.PC * BN < (1L << 22) && (long)s.L < (1L << 22) &&
           (long)s.KK < (1L << 22);
}

size_t lds_bytes(const RowsShape &s)
{
    const int BN = s.Cout > 32 ? 64 : 32;
    return ((size_t)s.x_floats + (size_t)(s.PC / 2) * (2 * BN + 2) + (size_t)s.PC) * sizeof(float);
}

}  // namespace

bool conv_rows_ok(const ConvRowsArgs &a)
{
    RowsShape s;
    return plan_rows(a, s);
}

bool conv_rows_preferred(const ConvRowsArgs &a)
{
    RowsShape s;
    return plan_rows(a, s) && s.nblk >= 4;
}

int conv_rows_tiles(const ConvRowsArgs &a)
{
    RowsShape s;
    if (!plan_rows(a, s)) return 0;
    return s.ktiles * s.ctiles;
}

void conv_rows_launch(const ConvRowsArgs &a, bool bf16, float scale, float *gW, float *gb, float *sqnorm,
                      float *partial, hipStream_t stream)
{
    RowsShape s;
    plan_rows(a, s);
    s.vec = s.KK % 4 == 0 && aligned(gW, 16);
    const int tiles = s.ktiles * s.ctiles;
    const int direct = tiles == 1;
    float *sqout = sqnorm ? (direct ? sqnorm : partial) : nullptr;
    const dim3 grid((unsigned)(a.N * tiles));
    const size_t lds = lds_bytes(s);
    if (s.Cout > 32) {
        if (bf16)
            conv_rows_kernel<uint16_t, 2><<<grid, kThreads, lds, stream>>>(
                (const uint16_t *)a.X, (const uint16_t *)a.GY, s, scale, gW, gb, sqout, direct);
        else
            conv_rows_kernel<float, 2><<<grid, kThreads, lds, stream>>>((const float *)a.X, (const float *)a.GY, s,
                                                                        scale, gW, gb, sqout, direct);
    } else {
        if (bf16)
            conv_rows_kernel<uint16_t, 1><<<grid, kThreads, lds, stream>>>(
                (const uint16_t *)a.X, (const uint16_t *)a.GY, s, scale, gW, gb, sqout, direct);
        else
            conv_rows_kernel<float, 1><<<grid, kThreads, lds, stream>>>((const float *)a.X, (const float *)a.GY, s,
                                                                        scale, gW, gb, sqout, direct);
    }
    if (sqnorm && !direct) sum_partials(partial, a.N, tiles, sqnorm, stream);
}

}  // namespace dpg
