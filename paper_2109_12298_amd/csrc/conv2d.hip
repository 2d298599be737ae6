// Conv2d per-sample gradients by implicit im2col on MFMA.
//
// For sample n the weight gradient is the product of the output backprop
// GY_n [Cout][L] (L = Ho*Wo positions) with the transposed unfold of the
// input, U_n [L][Cin*kh*kw], whose column kk = (ci, u, v) at position
// p = (oh, ow) is X_n[ci][oh*sh+u-ph][ow*sw+v-pw] (zero in the padding).
// The unfold is never formed, in HBM or in LDS.
//
// Fast path: a workgroup owns one (sample, kk-tile, co-tile).  It stages the
// input planes its kk-tile touches once, with a zero halo, in LDS; every
// unfold element is then one LDS read at (per-lane kk offset) + (per-position
// offset from a small table).  The MFMA "rows" run over kk, which is the
// contiguous index of the weight, so each lane ends holding four consecutive
// gradient entries and stores them as one float4.  The four waves split the
// output tile and/or the position (K) range; K-split partial tiles are added
// in LDS in wave order.  A sample whose gradient fits in one tile gets its
// squared norm written directly; otherwise tile partials go to the workspace
// and a second kernel adds them in tile order.
//
// Fallback (input planes too large for LDS): the same contraction with the
// unfold gathered through the cache into a K-major LDS tile per chunk.
#include "common.hpp"
#include "mfma_tile.hpp"
#include "conv2d_small.hpp"
#include "conv2d_rows.hpp"

#include <type_traits>

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kLdsBudget = 60 * 1024;   // dynamic LDS per workgroup (static arrays come on top)
constexpr int kStage = 8;               // global loads in flight per thread while staging

struct ConvShape {
    int Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
    int L, KK, khw;
};

// ---------------------------------------------------------------------------
// fast path
// ---------------------------------------------------------------------------
template <int FM, int FN, int WM, int WN, int WK>
struct ConvTile {
    static_assert(WM * WN * WK == 4 || WM * WN * WK == 8, "four or eight waves");
    static_assert((WK & (WK - 1)) == 0, "K split is a power of two");
    static constexpr int NT = 64 * WM * WN * WK;   // threads
    static constexpr int BM = WM * FM * 32;   // kk
    static constexpr int BN = WN * FN * 32;   // co
    static constexpr int LDG = BN + 1;        // padded row of the staged backprop chunk
};

struct ConvGeom {
    int Hp, Wp, plane;   // padded input plane
    int nplanes;         // planes staged per workgroup (upper bound)
    int tiles_m, tiles_n, tiles;
    int vec;             // float4 stores allowed (KK % 4 == 0 and gW 16-byte aligned)
    int bk;              // positions per staged chunk (multiple of 8)
    int one;             // whole sample staged with one load per register (see kOneX, kOneG)
    int xvec, gvec;      // one-shot staging may use float4 loads of X / GY
    int rowstep;         // sh * Wp: padded-plane offset of one output row
    float inv_plane, inv_wp, inv_bk, inv_wo, inv_hw, inv_w, inv_l;   // reciprocals for divmod
};

// elements per thread held in registers by the one-shot staging
constexpr int kOneX = 16;
constexpr int kOneG = 16;

// q = x / d, r = x % d for 0 <= x < 2^22 via a float reciprocal, corrected to
// the exact quotient without branches (the float estimate is off by at most one)
__device__ __forceinline__ void divmod(int x, int d, float inv_d, int &q, int &r)
{
    q = (int)((float)x * inv_d);
    r = x - q * d;
    q += (r >= d ? 1 : 0) - (r < 0 ? 1 : 0);
    r = x - q * d;
}

// Flat element held in register j by thread tid of a one-shot load.
template <int NT>
__device__ __forceinline__ int flat_at(int j, int tid, bool vec)
{
    return vec ? 4 * (tid + (j >> 2) * NT) + (j & 3) : tid + j * NT;
}

// Loads elements [0, count) of src (count >= 1) into registers, all loads
// issued before any is used; addresses past the end are clamped and their
// values zeroed, so there is no branch.  vec: float4 loads (count % 4 == 0,
// src 16-byte aligned).
template <int EPT, int NT, typename T>
__device__ __forceinline__ void flat_load(const T *__restrict__ src, int count, bool vec, int tid, float (&v)[EPT])
{
    if constexpr (std::is_same<T, float>::value) {
        if (vec) {
#pragma unroll
            for (int j = 0; j < EPT / 4; ++j) {
                const int e = 4 * (tid + j * NT);
                const int ec = e < count ? e : count - 4;
                const float4 q = *reinterpret_cast<const float4 *>(src + ec);
                const bool ok = e < count;
                v[4 * j + 0] = ok ? q.x : 0.0f;
                v[4 * j + 1] = ok ? q.y : 0.0f;
                v[4 * j + 2] = ok ? q.z : 0.0f;
                v[4 * j + 3] = ok ? q.w : 0.0f;
            }
            return;
        }
    }
#pragma unroll
    for (int j = 0; j < EPT; ++j) {
        const int e = tid + j * NT;
        const float x = load_elem<T>(src, e < count ? e : count - 1);
        v[j] = e < count ? x : 0.0f;
    }
}

template <typename T, int FM, int FN, int WM, int WN, int WK>
__global__ __launch_bounds__(64 * WM * WN * WK) void conv_per_sample_kernel(
    const T *__restrict__ X, const T *__restrict__ GY, ConvShape s, ConvGeom g, float scale,
    float *__restrict__ gW, float *__restrict__ gb, float *__restrict__ sqout, int direct)
{
    using Cfg = ConvTile<FM, FN, WM, WN, WK>;
    constexpr int NT = Cfg::NT;
    extern __shared__ float lds[];
    __shared__ float red16[16];
    __shared__ float bpart[NT];

    const i64 bsw = xcd_swizzle(blockIdx.x, gridDim.x);
    const int n = (int)(bsw / g.tiles);
    const int tile = (int)(bsw % g.tiles);
    const int tm = tile / g.tiles_n, tn = tile % g.tiles_n;
    const int m0 = tm * Cfg::BM;   // first kk
    const int n0 = tn * Cfg::BN;   // first co
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wk = wave % WK;
    const int wmn = wave / WK;
    const int wm = wmn % WM, wn = wmn / WM;

    const int BK = g.bk;
    float *Xs = lds;
    float *Gs = lds + g.nplanes * g.plane;

    const int ci0 = m0 / s.khw;
    int ci1 = (m0 + Cfg::BM - 1) / s.khw + 1;
    if (ci1 > s.Cin) ci1 = s.Cin;
    const int np = ci1 - ci0;
    const int nco = s.Cout - n0 < Cfg::BN ? s.Cout - n0 : Cfg::BN;
    const int HW = s.H * s.W;
    const T *Xn = X + (i64)n * s.Cin * HW;
    const T *Gn = GY + (i64)n * s.Cout * s.L;
    const bool pad = (s.ph | s.pw) != 0;

    if (g.one) {
        // ---- whole sample in one round trip: every load of X and GY is in
        // flight before the first is written to LDS
        float xv[kOneX], gv[kOneG];
        const int xcount = np * HW, gcount = nco * s.L;
        flat_load<kOneX, NT>(Xn + (i64)ci0 * HW, xcount, g.xvec != 0, tid, xv);
        flat_load<kOneG, NT>(Gn + (i64)n0 * s.L, gcount, g.gvec != 0, tid, gv);
        if (pad) {   // zero halo (disjoint from the interior written below)
            float *trash = Gs + BK * Cfg::LDG;
            for (int idx = tid; idx < np * g.plane; idx += NT) {
                int c, rem, r, q;
                divmod(idx, g.plane, g.inv_plane, c, rem);
                divmod(rem, g.Wp, g.inv_wp, r, q);
                const bool halo = r < s.ph || r >= s.ph + s.H || q < s.pw || q >= s.pw + s.W;
                *(halo ? Xs + idx : trash + lane) = 0.0f;
            }
        }
        if ((s.L & 1) && tid < Cfg::BN) Gs[s.L * Cfg::LDG + tid] = 0.0f;   // odd tail of the last position pair
        // registers past the end go to this lane's slot of a trash row
        float *trash = Gs + BK * Cfg::LDG;
#pragma unroll
        for (int j = 0; j < kOneX; ++j) {
            const int e = flat_at<NT>(j, tid, g.xvec != 0);
            int c, rem, ih, iw;
            divmod(e, HW, g.inv_hw, c, rem);
            divmod(rem, s.W, g.inv_w, ih, iw);
            float *dst = e < xcount ? Xs + c * g.plane + (ih + s.ph) * g.Wp + iw + s.pw : trash + lane;
            *dst = xv[j];
        }
#pragma unroll
        for (int j = 0; j < kOneG; ++j) {
            const int e = flat_at<NT>(j, tid, g.gvec != 0);
            int co, p;
            divmod(e, s.L, g.inv_l, co, p);
            float *dst = e < gcount ? Gs + p * Cfg::LDG + co : trash + lane;
            *dst = gv[j];
        }
    } else {
        // ---- stage the input planes this kk-tile reads, zero halo included;
        // kStage loads in flight per thread before any is written to LDS
        const int xtotal = np * g.plane;
        const T *Xc = Xn + (i64)ci0 * HW;
        float *trash = Gs + BK * Cfg::LDG;
        for (int i0 = tid; i0 < xtotal; i0 += NT * kStage) {
            float v[kStage];
#pragma unroll
            for (int j = 0; j < kStage; ++j) {
                const int idx = i0 + j * NT;
                int c, rem, r, q;
                divmod(idx, g.plane, g.inv_plane, c, rem);
                divmod(rem, g.Wp, g.inv_wp, r, q);
                const int ih = r - s.ph, iw = q - s.pw;
                const bool in = idx < xtotal && ih >= 0 && ih < s.H && iw >= 0 && iw < s.W;
                const float x = load_elem<T>(Xc, in ? (c * s.H + ih) * s.W + iw : 0);
                v[j] = in ? x : 0.0f;
            }
#pragma unroll
            for (int j = 0; j < kStage; ++j) {
                const int idx = i0 + j * NT;
                *(idx < xtotal ? Xs + idx : trash + lane) = v[j];
            }
        }
    }

    // ---- per-lane unfold column offsets
    int offkk[FM];
    bool vkk[FM];
#pragma unroll
    for (int x = 0; x < FM; ++x) {
        const int kk = m0 + wm * FM * 32 + x * 32 + (lane & 31);
        vkk[x] = kk < s.KK;
        const int k2 = vkk[x] ? kk : 0;
        const int ci = k2 / s.khw;
        const int rem = k2 - ci * s.khw;
        const int u = rem / s.kw;
        const int v = rem - u * s.kw;
        offkk[x] = vkk[x] ? (ci - ci0) * g.plane + u * g.Wp + v : 0;
    }

    f32x16 acc[FM][FN];
#pragma unroll
    for (int x = 0; x < FM; ++x)
#pragma unroll
        for (int y = 0; y < FN; ++y)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.0f;

    // bias: thread (seg, co) adds positions seg, seg + nseg, ... of each chunk
    const bool do_bias = gb != nullptr && tm == 0;
    constexpr int kSeg = NT / Cfg::BN;
    const int bco = tid % Cfg::BN, bseg = tid / Cfg::BN;
    float bias_acc = 0.0f;

    for (int p0 = 0; p0 < s.L; p0 += BK) {
        if (!g.one) {
            if (p0 > 0) __syncthreads();   // previous chunk fully consumed
            const int gtotal = Cfg::BN * BK;
            const T *Gc = Gn + (i64)n0 * s.L + p0;
            float *trash = Gs + BK * Cfg::LDG;
            for (int e0 = tid; e0 < gtotal; e0 += NT * kStage) {
                float v[kStage];
                float *at[kStage];
#pragma unroll
                for (int j = 0; j < kStage; ++j) {
                    const int e = e0 + j * NT;
                    int co, p;
                    divmod(e, BK, g.inv_bk, co, p);
                    at[j] = e < gtotal ? Gs + p * Cfg::LDG + co : trash + lane;
                    const bool in = e < gtotal && co < nco && p0 + p < s.L;
                    const float x = load_elem<T>(Gc, in ? co * s.L + p : 0);
                    v[j] = in ? x : 0.0f;
                }
#pragma unroll
                for (int j = 0; j < kStage; ++j) *at[j] = v[j];
            }
        }
        __syncthreads();
        const int len = s.L - p0 < BK ? s.L - p0 : BK;
        const int kpairs = (len + 1) >> 1;
        // two position pairs per trip (the second masked to zero past the
        // end) so that the LDS reads of both are issued before the MFMAs
        for (int q0 = wk; q0 < kpairs; q0 += 2 * WK) {
            float a[2][FM], b[2][FN];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const bool ok = q0 + h * WK < kpairs;
                const int ks = ok ? 2 * (q0 + h * WK) + (lane >> 5) : 0;
                int oh, ow;
                divmod(p0 + ks, s.Wo, g.inv_wo, oh, ow);
                const int op = ks < len ? oh * g.rowstep + ow * s.sw : 0;
#pragma unroll
                for (int x = 0; x < FM; ++x) a[h][x] = vkk[x] ? Xs[offkk[x] + op] : 0.0f;
#pragma unroll
                for (int y = 0; y < FN; ++y) {
                    const float v = Gs[ks * Cfg::LDG + wn * FN * 32 + y * 32 + (lane & 31)];
                    b[h][y] = ok ? v : 0.0f;
                }
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int x = 0; x < FM; ++x)
#pragma unroll
                    for (int y = 0; y < FN; ++y)
                        acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[h][x], b[h][y], acc[x][y], 0, 0, 0);
        }
        if (do_bias) {
            for (int p = bseg; p < len; p += kSeg) bias_acc += Gs[p * Cfg::LDG + bco];
        }
    }

    // ---- add the K-split partial tiles pairwise in a fixed tree (wave k
    // takes wave k + w/2), reusing the staging LDS
    if (WK > 1) {
        constexpr int kTile = FM * FN * 16 * 64;   // floats of one wave's accumulators
        float *R = lds;
#pragma unroll
        for (int w = WK; w > 1; w >>= 1) {
            const int half = w >> 1;
            __syncthreads();
            if (wk >= half && wk < w) {
                float *dst = R + ((wk - half) * WM * WN + wmn) * kTile;
#pragma unroll
                for (int x = 0; x < FM; ++x)
#pragma unroll
                    for (int y = 0; y < FN; ++y)
#pragma unroll
                        for (int r = 0; r < 16; ++r) dst[((x * FN + y) * 16 + r) * 64 + lane] = acc[x][y][r];
            }
            __syncthreads();
            if (wk < half) {
                const float *src = R + (wk * WM * WN + wmn) * kTile;
#pragma unroll
                for (int x = 0; x < FM; ++x)
#pragma unroll
                    for (int y = 0; y < FN; ++y)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[x][y][r] += src[((x * FN + y) * 16 + r) * 64 + lane];
            }
        }
    }

    float sq = 0.0f;
    if (wk == 0) {
        const bool vec = g.vec != 0;
        float *G = gW + (i64)n * s.Cout * s.KK;
#pragma unroll
        for (int x = 0; x < FM; ++x)
#pragma unroll
            for (int y = 0; y < FN; ++y) {
                const int co = n0 + wn * FN * 32 + y * 32 + (lane & 31);
                if (co >= s.Cout) continue;
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const int kk = m0 + wm * FM * 32 + x * 32 + 8 * rb + 4 * (lane >> 5);
                    const float g0 = scale * acc[x][y][4 * rb + 0], g1 = scale * acc[x][y][4 * rb + 1];
                    const float g2 = scale * acc[x][y][4 * rb + 2], g3 = scale * acc[x][y][4 * rb + 3];
                    float *dst = G + (i64)co * s.KK + kk;
                    if (vec && kk + 3 < s.KK) {
                        *reinterpret_cast<float4 *>(dst) = make_float4(g0, g1, g2, g3);
                        sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
                    } else {
                        if (kk + 0 < s.KK) { dst[0] = g0; sq += g0 * g0; }
                        if (kk + 1 < s.KK) { dst[1] = g1; sq += g1 * g1; }
                        if (kk + 2 < s.KK) { dst[2] = g2; sq += g2 * g2; }
                        if (kk + 3 < s.KK) { dst[3] = g3; sq += g3 * g3; }
                    }
                }
            }
    }
    if (do_bias) {   // segments added in order
        bpart[tid] = bias_acc;
        __syncthreads();
        if (tid < nco) {
            float b = 0.0f;
#pragma unroll
            for (int k = 0; k < kSeg; ++k) b += bpart[k * Cfg::BN + tid];
            const float v = scale * b;
            gb[(i64)n * s.Cout + n0 + tid] = v;
            sq += v * v;
        }
    }
    sq = block_sum(sq, red16);
    if (sqout && tid == 0) {
        if (direct) sqout[n] = sq;
        else sqout[(i64)n * g.tiles + tile] = sq;
    }
}

// ---------------------------------------------------------------------------
// fallback: unfold gathered per chunk through the cache
// ---------------------------------------------------------------------------
constexpr int kGM = 64, kGN = 64, kGK = 32;

template <typename T>
__global__ __launch_bounds__(kThreads) void conv_generic_kernel(
    const T *__restrict__ X, const T *__restrict__ GY, ConvShape s, int tiles_n, int tiles,
    float scale, float *__restrict__ gW, float *__restrict__ gb, float *__restrict__ sqout,
    int direct)
{
    __shared__ float As[kGK * kGM];   // [p][co]
    __shared__ float Bs[kGK * kGN];   // [p][kk]
    __shared__ float red[16];
    const int n = blockIdx.x / tiles;
    const int tile = blockIdx.x % tiles;
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const int m0 = tm * kGM, n0 = tn * kGN;    // m: co, n: kk
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * (kGM / 2), wn = (wave & 1) * (kGN / 2);
    const T *Xn = X + (i64)n * s.Cin * s.H * s.W;
    const T *Gn = GY + (i64)n * s.Cout * s.L;
    const bool do_bias = gb != nullptr && tn == 0;

    MfmaTile<kGM, kGN> t;
    t.zero();
    float bias_acc = 0.0f;
    for (int k0 = 0; k0 < s.L; k0 += kGK) {
        for (int e = tid; e < kGK * kGM; e += kThreads) {
            const int ii = e / kGK, kk = e % kGK;
            const int p = k0 + kk, co = m0 + ii;
            As[kk * kGM + ii] = (p < s.L && co < s.Cout) ? load_elem<T>(Gn, (i64)co * s.L + p) : 0.0f;
        }
        for (int e = tid; e < kGK * kGN; e += kThreads) {
            const int jj = e / kGK, kk = e % kGK;
            const int p = k0 + kk, j = n0 + jj;
            float v = 0.0f;
            if (p < s.L && j < s.KK) {
                const int ci = j / s.khw, rem = j - ci * s.khw;
                const int u = rem / s.kw, vv = rem - u * s.kw;
                const int oh = p / s.Wo, ow = p - oh * s.Wo;
                const int ih = oh * s.sh + u - s.ph, iw = ow * s.sw + vv - s.pw;
                if (ih >= 0 && ih < s.H && iw >= 0 && iw < s.W)
                    v = load_elem<T>(Xn, ((i64)ci * s.H + ih) * s.W + iw);
            }
            Bs[kk * kGN + jj] = v;
        }
        __syncthreads();
        t.template mma<kGK>(As, kGM, Bs, kGN, wm, wn, lane);
        if (do_bias && tid < kGM) {
            for (int kk = 0; kk < kGK; ++kk) bias_acc += As[kk * kGM + tid];
        }
        __syncthreads();
    }
    float sq = 0.0f;
    float *G = gW + (i64)n * s.Cout * s.KK;
    t.for_each(wm, wn, lane, [&](int r, int c, float v) {
        const int co = m0 + r, kk = n0 + c;
        if (co < s.Cout && kk < s.KK) {
            const float gv = scale * v;
            G[(i64)co * s.KK + kk] = gv;
            sq += gv * gv;
        }
    });
    if (do_bias && tid < kGM && m0 + tid < s.Cout) {
        const float v = scale * bias_acc;
        gb[(i64)n * s.Cout + m0 + tid] = v;
        sq += v * v;
    }
    sq = block_sum(sq, red);
    if (sqout && tid == 0) {
        if (direct) sqout[n] = sq;
        else sqout[(i64)n * tiles + tile] = sq;
    }
}

// ---------------------------------------------------------------------------
// host: pick a tile configuration
// ---------------------------------------------------------------------------
struct Plan {
    int cfg;                 // index into kConfigs, or -1 for the fallback
    ConvGeom g;
    size_t lds;
};

struct CfgDesc {
    int FM, FN, WM, WN, WK;
};

constexpr CfgDesc kConfigs[] = {
    {1, 1, 1, 1, 4},   // 32 x 32
    {2, 1, 1, 1, 4},   // 64 x 32
    {1, 2, 1, 1, 4},   // 32 x 64
    {2, 2, 1, 1, 4},   // 64 x 64
    {2, 1, 2, 1, 2},   // 128 x 32
    {2, 1, 4, 1, 1},   // 256 x 32
    {2, 2, 2, 1, 2},   // 128 x 64
    {2, 2, 2, 2, 1},   // 128 x 128
    {2, 2, 1, 2, 2},   // 64 x 128
    // eight waves: for grids too small to fill the chip with four-wave blocks
    {1, 1, 1, 1, 8},   // 32 x 32
    {2, 1, 1, 1, 8},   // 64 x 32
    {2, 1, 2, 1, 4},   // 128 x 32
    {2, 1, 4, 1, 2},   // 256 x 32
};
constexpr int kNumConfigs = sizeof(kConfigs) / sizeof(kConfigs[0]);
static_assert(kNumConfigs == 13, "dispatch_fast lists every configuration");

ConvGeom geom_for(const CfgDesc &c, const ConvShape &s)
{
    ConvGeom g;
    g.Hp = s.H + 2 * s.ph;
    g.Wp = s.W + 2 * s.pw;
    g.plane = g.Hp * g.Wp;
    const int BM = c.WM * c.FM * 32, BN = c.WN * c.FN * 32;
    int np = (BM - 1) / s.khw + 2;
    if (np > s.Cin) np = s.Cin;
    g.nplanes = np;
    g.tiles_m = (s.KK + BM - 1) / BM;
    g.tiles_n = (s.Cout + BN - 1) / BN;
    g.tiles = g.tiles_m * g.tiles_n;
    g.vec = 0;
    g.one = g.xvec = g.gvec = 0;
    return g;
}

// Positions per staged chunk: the whole sample when it fits (one load round
// trip), else as many as the LDS budget allows; a multiple of 8, at least 64.
int chunk_for(const CfgDesc &c, const ConvGeom &g, const ConvShape &s)
{
    const int BN = c.WN * c.FN * 32;
    const long avail = (long)kLdsBudget / 4 - (long)g.nplanes * g.plane - 64;
    long bk = avail / (BN + 1);
    bk &= ~7L;
    const int need = (s.L + 7) & ~7;
    if (bk > need) bk = need;
    if (bk < 64) bk = need < 64 ? need : 64;
    return (int)bk;
}

int threads_of(const CfgDesc &c) { return 64 * c.WM * c.WN * c.WK; }

size_t lds_for(const CfgDesc &c, const ConvGeom &g)
{
    const int BN = c.WN * c.FN * 32;
    const size_t stage = (size_t)g.nplanes * g.plane + (size_t)g.bk * (BN + 1) + 64;
    const size_t redf = (size_t)(c.WK / 2) * c.WM * c.WN * c.FM * c.FN * 16 * 64;
    return (stage > redf ? stage : redf) * sizeof(float);
}

// Grids of at most this many workgroups leave CUs idle or nearly so; their
// blocks get eight waves, so that each wave's serial share of the sample is
// halved and two waves per SIMD hide each other's latencies.
constexpr long kSmallGrid = 512;

Plan plan_conv(const ConvShape &s, long N)
{
    Plan best;
    best.cfg = -1;
    double best_cost = 0;
    for (int i = 0; i < kNumConfigs; ++i) {
        const CfgDesc &c = kConfigs[i];
        ConvGeom g = geom_for(c, s);
        g.bk = chunk_for(c, g, s);
        const size_t lds = lds_for(c, g);
        if (lds > (size_t)kLdsBudget) continue;
        const int BM = c.WM * c.FM * 32, BN = c.WN * c.FN * 32;
        // padded MFMA area, plus the re-staging of input planes per tile
        const double area = (double)g.tiles_m * BM * g.tiles_n * BN;
        const double stage = (double)g.tiles * g.nplanes * g.plane / 8.0;
        double cost = area + stage + (g.tiles > 1 ? 2048.0 : 0.0);
        const bool small = N * g.tiles <= kSmallGrid;
        if (threads_of(c) == 512) cost *= small ? 0.7 : 1.05;
        if (best.cfg < 0 || cost < best_cost) {
            best.cfg = i;
            best.g = g;
            best.lds = lds;
            best_cost = cost;
        }
    }
    return best;
}

template <typename T, int FM, int FN, int WM, int WN, int WK>
void launch_fast(const void *X, const void *GY, const ConvShape &s, const Plan &p, i64 N, float scale,
                 float *gW, float *gb, float *sqout, int direct, hipStream_t stream)
{
    conv_per_sample_kernel<T, FM, FN, WM, WN, WK><<<(unsigned)(N * p.g.tiles), 64 * WM * WN * WK, p.lds, stream>>>(
        (const T *)X, (const T *)GY, s, p.g, scale, gW, gb, sqout, direct);
}

template <typename T>
void dispatch_fast(const void *X, const void *GY, const ConvShape &s, const Plan &p, i64 N, float scale,
                   float *gW, float *gb, float *sqout, int direct, hipStream_t stream)
{
    switch (p.cfg) {
    case 0: launch_fast<T, 1, 1, 1, 1, 4>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 1: launch_fast<T, 2, 1, 1, 1, 4>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 2: launch_fast<T, 1, 2, 1, 1, 4>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 3: launch_fast<T, 2, 2, 1, 1, 4>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 4: launch_fast<T, 2, 1, 2, 1, 2>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 5: launch_fast<T, 2, 1, 4, 1, 1>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 6: launch_fast<T, 2, 2, 2, 1, 2>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 7: launch_fast<T, 2, 2, 2, 2, 1>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 8: launch_fast<T, 2, 2, 1, 2, 2>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 9: launch_fast<T, 1, 1, 1, 1, 8>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 10: launch_fast<T, 2, 1, 1, 1, 8>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    case 11: launch_fast<T, 2, 1, 2, 1, 4>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    default: launch_fast<T, 2, 1, 4, 1, 2>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream); break;
    }
}

int conv_tiles(const ConvShape &s, long N)
{
    const Plan p = plan_conv(s, N);
    if (p.cfg >= 0) return p.g.tiles;
    return ((s.KK + kGN - 1) / kGN) * ((s.Cout + kGM - 1) / kGM);
}

bool fits_int32(i64 Cin, i64 H, i64 W, i64 Cout, i64 kh, i64 kw)
{
    const i64 lim = i64(1) << 30;
    return Cin * H * W < lim && Cout * H * W < lim && Cin * kh * kw < lim && (H + 2 * kh) * (W + 2 * kw) < lim;
}

}  // namespace
}  // namespace dpg

using namespace dpg;

static ConvShape make_shape(int64_t Cin, int64_t H, int64_t W, int64_t Cout, int64_t kh, int64_t kw,
                            int64_t sh, int64_t sw, int64_t ph, int64_t pw)
{
    ConvShape s;
    s.Cin = (int)Cin; s.H = (int)H; s.W = (int)W; s.Cout = (int)Cout; s.kh = (int)kh; s.kw = (int)kw;
    s.sh = (int)sh; s.sw = (int)sw; s.ph = (int)ph; s.pw = (int)pw;
    s.Ho = (int)((H + 2 * ph - kh) / sh + 1);
    s.Wo = (int)((W + 2 * pw - kw) / sw + 1);
    s.L = s.Ho * s.Wo;
    s.khw = s.kh * s.kw;
    s.KK = s.Cin * s.khw;
    return s;
}

static bool shape_ok(int64_t Cin, int64_t H, int64_t W, int64_t Cout, int64_t kh, int64_t kw, int64_t sh,
                     int64_t sw, int64_t ph, int64_t pw)
{
    return Cin >= 1 && H >= 1 && W >= 1 && Cout >= 1 && kh >= 1 && kw >= 1 && sh >= 1 && sw >= 1 &&
           ph >= 0 && pw >= 0 && H + 2 * ph >= kh && W + 2 * pw >= kw;
}

extern "C" size_t dp_grad_sample_conv2d_workspace_bytes(int64_t N, int64_t Cin, int64_t H, int64_t W,
                                                        int64_t Cout, int64_t kh, int64_t kw, int64_t sh,
                                                        int64_t sw, int64_t ph, int64_t pw)
{
    if (N <= 0 || !shape_ok(Cin, H, W, Cout, kh, kw, sh, sw, ph, pw)) return 0;
    if (!fits_int32(Cin, H + 2 * ph, W + 2 * pw, Cout, kh, kw)) return 0;
    const ConvShape s = make_shape(Cin, H, W, Cout, kh, kw, sh, sw, ph, pw);
    const int tiles = conv_tiles(s, (long)N);
    // the row-chunked kernel's norm partials, when it has several tiles
    const ConvRowsArgs ra{nullptr, nullptr, N, Cin, H, W, Cout, (H + 2 * ph - kh) / sh + 1, (W + 2 * pw - kw) / sw + 1,
                          kh, kw, sh, sw, ph, pw};
    const int rtiles = conv_rows_tiles(ra);
    const int most = rtiles > tiles ? rtiles : tiles;
    return most > 1 ? (size_t)(N * most) * sizeof(float) : 0;
}

static int g_conv_path = DP_CONV_AUTO;

namespace dpg {
int conv_path()
{
    return g_conv_path;
}
}  // namespace dpg

extern "C" int dp_conv2d_set_path(int path)
{
    if (path != DP_CONV_AUTO && path != DP_CONV_TILED && path != DP_CONV_ROWS) return -1;
    const int prev = g_conv_path;
    g_conv_path = path;
    return prev;
}

extern "C" int32_t dp_conv2d_kernel_choice(int64_t N, int64_t Cin, int64_t H, int64_t W, int64_t Cout, int64_t kh,
                                           int64_t kw, int64_t sh, int64_t sw, int64_t ph, int64_t pw)
{
    if (N < 0 || !shape_ok(Cin, H, W, Cout, kh, kw, sh, sw, ph, pw)) return -1;
    if (!fits_int32(Cin, H + 2 * ph, W + 2 * pw, Cout, kh, kw)) return -1;
    const int64_t Ho = (H + 2 * ph - kh) / sh + 1, Wo = (W + 2 * pw - kw) / sw + 1;
    const ConvSmallArgs small{nullptr, nullptr, N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw};
    if (g_conv_path == DP_CONV_AUTO && conv_small_ok(small)) return DP_CONV_KERNEL_SMALL;
    const ConvRowsArgs rows{nullptr, nullptr, N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw};
    if (g_conv_path == DP_CONV_ROWS ? conv_rows_ok(rows) : g_conv_path == DP_CONV_AUTO && conv_rows_preferred(rows))
        return DP_CONV_KERNEL_ROWS;
    return DP_CONV_KERNEL_TILED;
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
    DPG_REQUIRE(fits_int32(Cin, H + 2 * ph, W + 2 * pw, Cout, kh, kw), DP_EUNSUPPORTED);
    DPG_REQUIRE(N == 0 || (X != nullptr && GY != nullptr && gW != nullptr), DP_EINVAL);
    const size_t need = dp_grad_sample_conv2d_workspace_bytes(N, Cin, H, W, Cout, kh, kw, sh, sw, ph, pw);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;

    const bool bf = dt == DP_BF16;
    const ConvSmallArgs small{X, GY, N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw};
    if (g_conv_path == DP_CONV_AUTO && conv_small_ok(small)) {
        // the whole sample fits one workgroup's LDS
        conv_small_launch(small, bf, scale, gW, gb, sqnorm, stream);
        return launch_status();
    }
    const ConvRowsArgs rows{X, GY, N, Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw};
    if (g_conv_path == DP_CONV_ROWS ? conv_rows_ok(rows) : g_conv_path == DP_CONV_AUTO && conv_rows_preferred(rows)) {
        // output row chunks, the whole weight-column tile in registers
        conv_rows_launch(rows, bf, scale, gW, gb, sqnorm, (float *)ws, stream);
        return launch_status();
    }
    const ConvShape s = make_shape(Cin, H, W, Cout, kh, kw, sh, sw, ph, pw);
    Plan p = plan_conv(s, (long)N);
    p.g.vec = (s.KK % 4 == 0) && aligned(gW, 16);
    if (p.cfg >= 0) {
        p.g.inv_plane = 1.0f / (float)p.g.plane;
        p.g.inv_wp = 1.0f / (float)p.g.Wp;
        p.g.inv_bk = 1.0f / (float)p.g.bk;
        p.g.inv_wo = 1.0f / (float)s.Wo;
        p.g.inv_hw = 1.0f / (float)(s.H * s.W);
        p.g.inv_w = 1.0f / (float)s.W;
        p.g.inv_l = 1.0f / (float)s.L;
        p.g.rowstep = s.sh * p.g.Wp;
        const CfgDesc &c = kConfigs[p.cfg];
        const long BN = c.WN * c.FN * 32;
        const long nt = threads_of(c);
        p.g.one = p.g.bk >= s.L && (long)p.g.nplanes * s.H * s.W <= nt * kOneX && BN * s.L <= nt * kOneG;
        p.g.xvec = !bf && (s.H * s.W) % 4 == 0 && aligned(X, 16);
        p.g.gvec = !bf && ((long)s.Cout * s.L) % 4 == 0 && aligned(GY, 16);
    }
    const int tiles = p.cfg >= 0 ? p.g.tiles : conv_tiles(s, (long)N);
    const int direct = tiles == 1;
    float *sqout = sqnorm ? (direct ? sqnorm : (float *)ws) : nullptr;
    if (p.cfg >= 0) {
        if (bf) dispatch_fast<uint16_t>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream);
        else dispatch_fast<float>(X, GY, s, p, N, scale, gW, gb, sqout, direct, stream);
    } else {
        const int tiles_n = (s.KK + kGN - 1) / kGN;
        const dim3 grid((unsigned)(N * tiles));
        if (bf)
            conv_generic_kernel<uint16_t><<<grid, kThreads, 0, stream>>>((const uint16_t *)X, (const uint16_t *)GY,
                                                                       s, tiles_n, tiles, scale, gW, gb, sqout,
                                                                       direct);
        else
            conv_generic_kernel<float><<<grid, kThreads, 0, stream>>>((const float *)X, (const float *)GY, s,
                                                                    tiles_n, tiles, scale, gW, gb, sqout, direct);
    }
    if (sqnorm && !direct)
        sum_partials((const float *)ws, N, tiles, sqnorm, stream);
    return launch_status();
}
