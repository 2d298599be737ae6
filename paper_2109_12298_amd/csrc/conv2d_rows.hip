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
// chunks.  Per chunk it loads the input rows the chunk reads (the tile's input
// channels) and the chunk's backprop into registers, all loads in flight at
// once, writes them to LDS, and contracts over the chunk's positions on
// v_mfma_f32_32x32x2_f32: per position pair a lane reads one unfold element
// per block (its column's offset plus the position's, from a table) and one
// backprop element, and the same position work feeds four or five MFMAs.
// Against tiling the unfold by columns and staging whole planes, this stages
// each backprop element once per column tile instead of once per 32 columns,
// and keeps the index arithmetic per MFMA small.
//
// LDS banks.  The staged input has a row stride = kw and a channel stride =
// kh * kw (mod 32), so the 32 consecutive unfold columns a half-wave reads
// land in 32 different banks whatever the kernel size; the backprop sits as
// [position pair][parity][channel], so each half-wave reads 32 consecutive
// channels, with an odd pair stride that spreads the staging writes.
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

struct RowsShape {
    int Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
    int Wp, L, KK, khw;
    int xR, xC;           // staged input: LDS floats per row and per channel
    int nblk;             // 32-column blocks per tile (<= 9)
    int ktiles, ctiles;   // column tiles, channel tiles
    int np;               // input channels a column tile touches (upper bound)
    int RC, XR;           // output rows per chunk, staged input rows per chunk
    int PC;               // positions per chunk, RC * Wo rounded up to even
    int x_floats;         // np * XR * Wp
    int vec;              // float4 stores of gW
    int fast;             // full tiles (nblk == kMaxBlk), stride 1, 16-byte runs: the branch-free contraction
    int xcd;              // a sample's tiles on one XCD (where a tile reads at least the bytes it stores)
    float inv_khw, inv_kw, inv_wo;
    // staging runs of VW elements: xwv = W / VW runs per input row, gqv =
    // PC / VW runs per channel of the chunk's backprop.  Stepping a run index
    // by kThreads: (channel, row, run) of the input by (xs_c, xs_r, xs_k),
    // (channel, run) of the backprop by (gs_c, gs_q); the global element
    // offsets and the LDS offsets follow by the step and wrap constants.
    int vw, xwv, gqv;
    int xs_c, xs_r, xs_k, gs_c, gs_q;
    int xg_step, xg_wrap_r, xl_step, xl_wrap_k, xl_wrap_r, gg_step, gg_wrap_q;
    float inv_xrw, inv_xwv, inv_gqv;
};

__device__ __forceinline__ void fdivmod(int x, int d, float inv_d, int &q, int &r)
{
    q = (int)((float)x * inv_d);
    r = x - q * d;
    q += (r >= d ? 1 : 0) - (r < 0 ? 1 : 0);
    r = x - q * d;
}

// Raw-buffer loads over one sample's tensor: 32-bit byte offsets, and an
// offset past the buffer's size reads zero (the zero halo and everything past
// the chunk or the tile come from that, with no branch and no mask).
constexpr uint32_t kOutside = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t sample_buffer(const void *base, uint32_t bytes)
{
    // 0x00020000: the gfx9 descriptor word for 32-bit untyped accesses
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, 0x00020000);
}

// XW dwords of raw data: VW elements of T (one bf16 element sits in the low
// half of its dword)
template <int XW>
struct Raw {
    uint32_t w[XW];
};

template <typename T, int VW, int XW>
__device__ __forceinline__ Raw<XW> raw_load_v(__amdgpu_buffer_rsrc_t r, uint32_t byte_off)
{
    Raw<XW> x;
    if constexpr (XW == 4) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0);
        x.w[0] = v[0]; x.w[1] = v[1]; x.w[2] = v[2]; x.w[3] = v[3];
    } else if constexpr (XW == 2) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, byte_off, 0, 0);
        x.w[0] = v[0]; x.w[1] = v[1];
    } else if constexpr (sizeof(T) == 4) {
        x.w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0);
    } else {
        x.w[0] = __builtin_amdgcn_raw_buffer_load_b16(r, byte_off, 0, 0);
    }
    return x;
}

template <typename T, int VW, int XW>
__device__ __forceinline__ void unpack(const Raw<XW> &x, float (&v)[VW])
{
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int t = 0; t < VW; ++t) v[t] = __builtin_bit_cast(float, x.w[t]);
    } else if constexpr (VW == 1) {
        v[0] = __builtin_bit_cast(float, x.w[0] << 16);
    } else {
#pragma unroll
        for (int t = 0; t < VW; ++t)
            v[t] = __builtin_bit_cast(float, (t & 1) ? (x.w[t >> 1] & 0xFFFF0000u) : (x.w[t >> 1] << 16));
    }
}

// The contraction of a chunk for full tiles at stride 1 (Wo a multiple of 4,
// so the chunk holds whole groups of four positions and the four positions
// 4k .. 4k+3 sit in one output row): the wave's NACT blocks are compile-time,
// so the loop has no branch; pair q's position offset is pbase + half and
// pair q+1's two further, tracked in scalars instead of read from the
// position table, and each block's two operands are one ds_read2.  SHX is
// the block shared by the two wave rows (-1: none), whose MFMA wave row wq
// runs for pair q + wq of each step only (operands chosen by selects).  The
// accumulation order per block is the generic loop's (pair q, then q+1).
template <int FM, int NACT, int SHX, int BN>
__device__ __forceinline__ void contract_fast(f32x16_t (&acc)[FM], const int (&koff)[FM], const float *Xs,
                                              const float *Gs, int qfull, int half, int gl, int Wo, int xR, int wq)
{
    constexpr int GSP = 2 * BN + 1;
    const float *gp = Gs + half * BN + gl;
    int pbase = 0, ow0 = 0;
    for (int q = 0; q < qfull; q += 2) {
        const int po = pbase + half;
        float a0[NACT], a1[NACT];
#pragma unroll
        for (int x = 0; x < NACT; ++x) {
            const float *xp = Xs + koff[x] + po;
            a0[x] = xp[0];
            a1[x] = xp[2];
        }
        const float b0 = gp[q * GSP], b1 = gp[(q + 1) * GSP];
#pragma unroll
        for (int x = 0; x < NACT; ++x)
            if (x != SHX) acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[x], b0, acc[x], 0, 0, 0);
#pragma unroll
        for (int x = 0; x < NACT; ++x)
            if (x != SHX) acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[x], b1, acc[x], 0, 0, 0);
        if constexpr (SHX >= 0) {
            // the shared block: wave row wq takes pair q + wq of the two
            const float as = wq == 0 ? a0[SHX] : a1[SHX];
            const float bs = wq == 0 ? b0 : b1;
            acc[SHX] = __builtin_amdgcn_mfma_f32_32x32x2f32(as, bs, acc[SHX], 0, 0, 0);
        }
        ow0 += 4;
        pbase += 4;
        const bool wrap = ow0 == Wo;
        ow0 = wrap ? 0 : ow0;
        pbase += wrap ? xR - Wo : 0;
    }
}

// WCO: 32-channel blocks per tile (1 or 2).  The waves form (4 / WCO) column
// rows x WCO channel columns; wave row q takes blocks q, q + 4/WCO, ...
// VW: elements per staging load (4: a 16-byte run of an input row or of a
// channel's backprop; 1: single elements).  XS, GS: X and backprop loads per
// thread per chunk, at most.  OCC: workgroups per CU the registers allow.
template <typename T, int WCO, int VW, int XS, int GS, int OCC, bool FAST>
__global__ __launch_bounds__(kThreads, OCC) void conv_rows_kernel(const T *__restrict__ X, const T *__restrict__ GY,
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
    // a sample's tiles on one XCD, so that the input channels and backprop
    // rows that several of them read are served from that XCD's L2 (for
    // tiles whose stores outweigh their reads, spreading them measured better)
    const i64 bsw = s.xcd ? xcd_swizzle(blockIdx.x, gridDim.x) : (i64)blockIdx.x;
    const i64 n = bsw / tiles;
    const int tile = (int)(bsw % tiles);
    const int tk = tile / s.ctiles, tc = tile % s.ctiles;
    const int m0 = tk * s.nblk * 32;          // first weight column
    const int n0 = tc * BN;                   // first output channel
    const int ci0 = m0 / s.khw;
    const int tid = threadIdx.x, lane = tid & 63, half = lane >> 5;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wq = wave / WCO, wc = wave % WCO;
    float *Xs = lds;                                   // [np][XR][Wp]
    constexpr int GSP = 2 * BN + 1;                    // floats per position pair (odd: staging writes spread over banks)
    float *Gs = lds + s.x_floats;                      // [PC/2][2][BN], pair stride GSP
    int *Pt = reinterpret_cast<int *>(Gs + s.PC / 2 * GSP);   // [PC] offset of position p in the staged rows
    const T *Xn = X + n * (i64)s.Cin * s.H * s.W;
    const T *Gn = GY + n * (i64)s.Cout * s.L;
    const int cvalid = s.Cout - n0 < BN ? s.Cout - n0 : BN;

    // the lane's unfold column offsets in the staged rows (a column past the
    // tile or the weight reads offset 0; its output rows are never stored).
    // Wave row wq takes blocks wq, wq + WKK, ...; with two wave rows and an
    // odd block count the last block is shared: each wave row runs its MFMAs
    // for one of the two pairs of every step (h == wq), and the two partial
    // tiles are added before the store, so both rows carry nblk / 2 blocks.
    int koff[FM], blkx[FM];
    bool bon[FM], bsh[FM];
#pragma unroll
    for (int x = 0; x < FM; ++x) {
        int blk = wq + WKK * x;
        bsh[x] = WKK == 2 && (s.nblk & 1) && x == s.nblk / 2;
        if (bsh[x]) blk = s.nblk - 1;
        blkx[x] = blk;
        bon[x] = blk < s.nblk;
        const int kk = m0 + blk * 32 + (lane & 31);
        koff[x] = 0;
        if (bon[x] && kk < s.KK) {
            int ci, rem, u, v;
            fdivmod(kk, s.khw, s.inv_khw, ci, rem);
            fdivmod(rem, s.kw, s.inv_kw, u, v);
            koff[x] = (ci - ci0) * s.xC + u * s.xR + v;
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
    // ---- staging.  The input stage holds, per tile channel c < np and staged
    // row r < XR, the row's W data columns at LDS c * xC + r * xR + pw + w; the
    // halo columns are cleared once and never written again, rows outside the
    // input read zeros.  A load covers a run of VW consecutive elements: runs
    // (c, r, k) of W / VW, and of the backprop (channel co, run q of the
    // chunk's positions).  Thread t takes runs t, t + kThreads, ...; their
    // indices and offsets are stepped by constants, not divided out.  An
    // element outside the input, the chunk or the tile reads past the
    // sample's buffer, which gives zero; the loaded values are not touched
    // until the chunk is written to LDS, so every load stays in flight.
    const __amdgpu_buffer_rsrc_t xbuf = sample_buffer(Xn, (uint32_t)(s.Cin * s.H * s.W) * (uint32_t)sizeof(T));
    const __amdgpu_buffer_rsrc_t gbuf = sample_buffer(Gn, (uint32_t)(s.Cout * s.L) * (uint32_t)sizeof(T));
    constexpr int XW = VW * sizeof(T) / 4 > 0 ? VW * sizeof(T) / 4 : 1;   // dwords per X load (bf16 singles: 1)
    Raw<XW> xv[XS], gv[GS];
    const int xruns = s.np * s.XR * s.xwv;                 // X runs per chunk
    const int gruns = BN * s.gqv;                          // backprop runs per chunk
    const int cmax = s.Cin - ci0 < s.np ? s.Cin - ci0 : s.np;
    int xc0, xr0, xk0, gc0, gq0;
    {
        int rem;
        fdivmod(tid, s.XR * s.xwv, s.inv_xrw, xc0, rem);
        fdivmod(rem, s.xwv, s.inv_xwv, xr0, xk0);
        fdivmod(tid, s.gqv, s.inv_gqv, gc0, gq0);
    }
    // halo columns: cleared once (they are never loaded)
    if (s.pw > 0) {
        for (int i = tid; i < s.x_floats; i += kThreads) Xs[i] = 0.0f;
    }

    auto load_chunk = [&](int oh0) {
        const int rows = s.Ho - oh0 < s.RC ? s.Ho - oh0 : s.RC;
        const int len = rows * s.Wo;
        const int ih0 = oh0 * s.sh - s.ph;
        int c = xc0, r = xr0, k = xk0;
        int off = ((ci0 + c) * s.H + ih0 + r) * s.W + VW * k;      // element offset in the sample's input
#pragma unroll
        for (int j = 0; j < XS; ++j) {
            if (j * kThreads < xruns) {
                const bool in = (c < cmax) & ((unsigned)(ih0 + r) < (unsigned)s.H);
                xv[j] = raw_load_v<T, VW, XW>(xbuf, in ? (uint32_t)off * (uint32_t)sizeof(T) : kOutside);
                k += s.xs_k;
                if (k >= s.xwv) {
                    k -= s.xwv;
                    ++r;
                }
                r += s.xs_r;
                if (r >= s.XR) {
                    r -= s.XR;
                    ++c;
                    off += s.xg_wrap_r;
                }
                c += s.xs_c;
                off += s.xg_step;
            }
        }
        int co = gc0, q = gq0;
        int goff = (n0 + co) * s.L + oh0 * s.Wo + VW * q;
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            if (j * kThreads < gruns) {
                const bool in = (co < cvalid) & (VW * q < len);
                gv[j] = raw_load_v<T, VW, XW>(gbuf, in ? (uint32_t)goff * (uint32_t)sizeof(T) : kOutside);
                q += s.gs_q;
                if (q >= s.gqv) {
                    q -= s.gqv;
                    ++co;
                    goff += s.gg_wrap_q;
                }
                co += s.gs_c;
                goff += s.gg_step;
            }
        }
    };
    // ---- the loaded chunk into LDS: the input rows at c * xC + r * xR + pw +
    // w, the backprop as [pair][parity][channel]
    auto store_chunk = [&]() {
        // every load has landed: said once here (vmcnt 0, the other counters
        // untouched) so that no later write of these registers waits again
        __builtin_amdgcn_s_waitcnt(0x0F70);
        int c = xc0, r = xr0, k = xk0;
        int lo = c * s.xC + r * s.xR + s.pw + VW * k;
#pragma unroll
        for (int j = 0; j < XS; ++j) {
            if (j * kThreads < xruns) {
                if (c < s.np) {
                    float v[VW];
                    unpack<T, VW, XW>(xv[j], v);
#pragma unroll
                    for (int t = 0; t < VW; ++t) Xs[lo + t] = v[t];
                }
                k += s.xs_k;
                if (k >= s.xwv) {
                    k -= s.xwv;
                    ++r;
                    lo += s.xl_wrap_k;
                }
                r += s.xs_r;
                if (r >= s.XR) {
                    r -= s.XR;
                    ++c;
                    lo += s.xl_wrap_r;
                }
                c += s.xs_c;
                lo += s.xl_step;
            }
        }
        int co = gc0, q = gq0;
#pragma unroll
        for (int j = 0; j < GS; ++j) {
            if (j * kThreads < gruns) {
                if (co < BN) {
                    float v[VW];
                    unpack<T, VW, XW>(gv[j], v);
#pragma unroll
                    for (int t = 0; t < VW; ++t) {
                        const int p = VW * q + t;
                        Gs[(p >> 1) * GSP + (p & 1) * BN + co] = v[t];
                    }
                }
                q += s.gs_q;
                if (q >= s.gqv) {
                    q -= s.gqv;
                    ++co;
                }
                co += s.gs_c;
            }
        }
    };

    for (int oh0 = 0; oh0 < s.Ho; oh0 += s.RC) {
        const int rows = s.Ho - oh0 < s.RC ? s.Ho - oh0 : s.RC;
        const int len = rows * s.Wo;                   // positions of this chunk
        load_chunk(oh0);                               // in flight while the other waves finish
        __syncthreads();                               // the previous chunk is consumed
        store_chunk();
        if constexpr (!FAST) {
            for (int p = tid; p < s.PC; p += kThreads) {
                int oh, ow;
                fdivmod(p, s.Wo, s.inv_wo, oh, ow);
                Pt[p] = p < len ? oh * s.sh * s.xR + ow * s.sw : 0;
            }
        }
        __syncthreads();
        if (do_bias) {
            // thread (bseg, bco): positions bseg, bseg + kSegs, ... of the chunk, in order
            for (int p = bseg; p < len; p += kSegs) bacc += Gs[(p >> 1) * GSP + (p & 1) * BN + bco];
        }
        // ---- contraction over the chunk's position pairs; the next pair's
        // reads are issued before the current pair's MFMAs
        const int npairs = (len + 1) >> 1;
        const int gl = wc * 32 + (lane & 31);
        // whole pairs two at a time without masks, then what is left masked
        const int qfull = (len >> 2) << 1;
        if constexpr (FAST) {
            // (the chunk holds whole groups of four positions: no remainder)
            if constexpr (WKK == 2) {
                // nine blocks over two wave rows: five each, the last shared
                contract_fast<FM, 5, 4, BN>(acc, koff, Xs, Gs, qfull, half, gl, s.Wo, s.xR, wq);
            } else {
                // nine blocks over four wave rows: row 0 takes 0, 4, 8, the others two
                if (wq == 0) contract_fast<FM, 3, -1, BN>(acc, koff, Xs, Gs, qfull, half, gl, s.Wo, s.xR, wq);
                else contract_fast<FM, 2, -1, BN>(acc, koff, Xs, Gs, qfull, half, gl, s.Wo, s.xR, wq);
            }
            continue;
        }
        for (int q = 0; q < qfull; q += 2) {
            float a[2][FM], b[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int pr = q + h;
                const int po = Pt[2 * pr + half];
                b[h] = Gs[pr * GSP + half * BN + gl];
#pragma unroll
                for (int x = 0; x < FM; ++x)
                    if (!bsh[x] || h == wq) a[h][x] = Xs[koff[x] + po];
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int x = 0; x < FM; ++x)
                    if (bon[x] && (!bsh[x] || h == wq))
                        acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[h][x], b[h], acc[x], 0, 0, 0);
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
                const float bv = Gs[pr * GSP + half * BN + gl];
                b[h] = pin ? bv : 0.0f;
#pragma unroll
                for (int x = 0; x < FM; ++x) {
                    if (!bsh[x] || h == wq) {
                        const float av = Xs[koff[x] + po];
                        a[h][x] = pin ? av : 0.0f;
                    }
                }
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int x = 0; x < FM; ++x)
                    if (bon[x] && (!bsh[x] || h == wq))
                        acc[x] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[h][x], b[h], acc[x], 0, 0, 0);
        }
    }
    if (WKK == 2 && (s.nblk & 1)) {
        // the shared block: wave row 1 hands its partial tile to wave row 0
        // through LDS ([channel column][register][lane], 8 KB)
        __syncthreads();                               // the stage is consumed
        float *part = lds + wc * 16 * 64;
#pragma unroll
        for (int x = 0; x < FM; ++x)
            if (bsh[x] && wq == 1)
#pragma unroll
                for (int r = 0; r < 16; ++r) part[r * 64 + lane] = acc[x][r];
        __syncthreads();
#pragma unroll
        for (int x = 0; x < FM; ++x)
            if (bsh[x] && wq == 0)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[x][r] += part[r * 64 + lane];
    }

    // ---- store the tile and its squared norm
    float sq = 0.0f;
    const int co = n0 + wc * 32 + (lane & 31);
    float *G = gW + n * (i64)s.Cout * s.KK;
#pragma unroll
    for (int x = 0; x < FM; ++x) {
        if (!bon[x] || co >= s.Cout || (bsh[x] && wq != 0)) continue;
        const int kb = m0 + blkx[x] * 32;
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
    // LDS-only barriers from here on: a __syncthreads would also wait for the
    // gradient stores just issued, and hold the workgroup's slot until they land
    if (do_bias) {
        bsum[bseg * BN + bco] = bacc;
        lds_barrier();
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
    lds_barrier();
    if (tid == 0 && sqout) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += red[w];
        if (direct) sqout[n] = t;
        else sqout[n * tiles + tile] = t;
    }
}

// LDS strides of the staged input.  A 32-column block's unfold read has lane
// j at column kk0 + j, i.e. at ci * xC + u * xR + v for kk = (ci, u, v); with
// xR = kw and xC = kh * kw (mod 32) that is kk (mod 32) plus a constant, so the
// 32 lanes of a half-wave hit 32 different banks for any kernel size.
int row_stride(int Wp, int kw)
{
    return Wp + (((kw - Wp) % 32) + 32) % 32;
}

int chan_stride(int XR, int xR, int khw)
{
    const int d = XR * xR;
    return d + (((khw - d) % 32) + 32) % 32;
}

// Kernel variants: elements per staging load, loads per thread, workgroups
// per CU and the LDS budget that keeps them resident.
struct Variant {
    int vw, xs, gs, occ, lds;
};
constexpr Variant kLarge4{4, 8, 8, 2, 72 * 1024};     // 16-byte runs, two workgroups per CU
constexpr Variant kSmall4{4, 2, 2, 3, 50 * 1024};     // 16-byte runs, three workgroups per CU
constexpr Variant kSingle{1, 16, 16, 2, 72 * 1024};   // single elements (any shape)

// The row chunk and staging constants of a variant; false if no chunk fits.
bool plan_rows(const ConvRowsArgs &a, const Variant &v, RowsShape &s)
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
    s.vw = v.vw;
    if (v.vw > 1 && (s.W % v.vw != 0 || s.Wo % v.vw != 0)) return false;
    // the largest row chunk whose stage fits the LDS budget (np * xC + PC / 2
    // * (2 BN + 1) + PC floats) and the per-thread load registers
    const int BN = 32 * wco;
    s.RC = 0;
    for (int rc = s.Ho; rc >= 1; --rc) {
        const int xr = (rc - 1) * s.sh + s.kh;
        const int pc = (rc * s.Wo + 1) & ~1;
        const long xf = ((long)s.np * chan_stride(xr, row_stride(s.Wp, s.kw), s.khw) + 3) & ~3L;
        const long fl = xf + (long)pc / 2 * (2 * BN + 1) + pc;
        const bool regs = (long)s.np * xr * (s.W / v.vw) <= (long)v.xs * kThreads &&
                          (long)BN * (pc / v.vw) <= (long)v.gs * kThreads;
        if (fl * 4 <= v.lds && regs) {
            s.RC = rc;
            break;
        }
    }
    if (s.RC == 0) return false;
    s.XR = (s.RC - 1) * s.sh + s.kh;
    s.PC = (s.RC * s.Wo + 1) & ~1;
    s.xR = row_stride(s.Wp, s.kw);
    s.xC = chan_stride(s.XR, s.xR, s.khw);
    s.x_floats = (s.np * s.xC + 3) & ~3;      // the backprop stage starts 16-byte aligned
    s.vec = 0;
    s.fast = v.vw == 4 && s.nblk == kMaxBlk && s.sh == 1 && s.sw == 1 && s.Wo % 4 == 0;
    {
        // per tile: the input channels and backprop rows read, the gradient block stored
        const long reads = (long)s.np * s.H * s.W + (long)BN * s.L;
        const long writes = (long)s.nblk * 32 * BN;
        s.xcd = s.ktiles * s.ctiles > 1 && reads >= writes;
    }
    s.inv_khw = 1.0f / (float)s.khw;
    s.inv_kw = 1.0f / (float)s.kw;
    s.inv_wo = 1.0f / (float)s.Wo;
    s.xwv = s.W / v.vw;
    s.gqv = s.PC / v.vw;
    s.inv_xrw = 1.0f / (float)(s.XR * s.xwv);
    s.inv_xwv = 1.0f / (float)s.xwv;
    s.inv_gqv = 1.0f / (float)s.gqv;
    {
        const int rows = kThreads / s.xwv;
        s.xs_k = kThreads % s.xwv;
        s.xs_r = rows % s.XR;
        s.xs_c = rows / s.XR;
        s.gs_q = kThreads % s.gqv;
        s.gs_c = kThreads / s.gqv;
        const int hw = s.H * s.W;
        // input element offset ((ci0 + c) * H + ih0 + r) * W + VW * k: a run
        // wrap (k past the row, r + 1) leaves it unchanged
        s.xg_step = v.vw * s.xs_k + s.xs_r * s.W + s.xs_c * hw;
        s.xg_wrap_r = hw - s.XR * s.W;
        // LDS offset c * xC + r * xR + pw + VW * k
        s.xl_step = v.vw * s.xs_k + s.xs_r * s.xR + s.xs_c * s.xC;
        s.xl_wrap_k = s.xR - s.W;
        s.xl_wrap_r = s.xC - s.XR * s.xR;
        // backprop element offset (n0 + co) * L + oh0 * Wo + VW * q
        s.gg_step = v.vw * s.gs_q + s.gs_c * s.L;
        s.gg_wrap_q = s.L - v.vw * s.gqv;
    }
    // index arithmetic through float reciprocals needs values below 2^22
    return (long)s.x_floats < (1L << 22) && (long)s.PC * BN < (1L << 22) && (long)s.L < (1L << 22) &&
           (long)s.KK < (1L << 22) && (long)s.np * s.XR * s.W < (1L << 22);
}

size_t lds_bytes(const RowsShape &s)
{
    const int BN = s.Cout > 32 ? 64 : 32;
    const size_t b = ((size_t)s.x_floats + (size_t)(s.PC / 2) * (2 * BN + 1) + (size_t)s.PC) * sizeof(float);
    // two wave rows hand a shared block's partial tile over in 8 KB
    const size_t hand = BN == 64 ? 2 * 16 * 64 * sizeof(float) : 0;
    return b > hand ? b : hand;
}

template <typename T, int WCO, int VW, int XS, int GS, int OCC>
void launch_variant(const ConvRowsArgs &a, const RowsShape &s, float scale, float *gW, float *gb, float *sqout,
                    int direct, hipStream_t stream)
{
    const dim3 grid((unsigned)(a.N * s.ktiles * s.ctiles));
    if constexpr (VW == 4) {
        if (s.fast) {
            conv_rows_kernel<T, WCO, VW, XS, GS, OCC, true><<<grid, kThreads, lds_bytes(s), stream>>>(
                (const T *)a.X, (const T *)a.GY, s, scale, gW, gb, sqout, direct);
            return;
        }
    }
    conv_rows_kernel<T, WCO, VW, XS, GS, OCC, false><<<grid, kThreads, lds_bytes(s), stream>>>(
        (const T *)a.X, (const T *)a.GY, s, scale, gW, gb, sqout, direct);
}

template <typename T, int WCO>
void launch_typed(const ConvRowsArgs &a, int which, const RowsShape &s, float scale, float *gW, float *gb,
                  float *sqout, int direct, hipStream_t stream)
{
    if (which == 0)
        launch_variant<T, WCO, kLarge4.vw, kLarge4.xs, kLarge4.gs, kLarge4.occ>(a, s, scale, gW, gb, sqout, direct,
                                                                              stream);
    else if (which == 1)
        launch_variant<T, WCO, kSmall4.vw, kSmall4.xs, kSmall4.gs, kSmall4.occ>(a, s, scale, gW, gb, sqout, direct,
                                                                              stream);
    else
        launch_variant<T, WCO, kSingle.vw, kSingle.xs, kSingle.gs, kSingle.occ>(a, s, scale, gW, gb, sqout, direct,
                                                                              stream);
}

}  // namespace

bool conv_rows_ok(const ConvRowsArgs &a)
{
    RowsShape s;
    return plan_rows(a, kSingle, s);
}

bool conv_rows_preferred(const ConvRowsArgs &a)
{
    RowsShape s;
    return plan_rows(a, kSingle, s) && s.nblk >= 4;
}

int conv_rows_tiles(const ConvRowsArgs &a)
{
    RowsShape s;
    if (!plan_rows(a, kSingle, s)) return 0;
    return s.ktiles * s.ctiles;
}

void conv_rows_launch(const ConvRowsArgs &a, bool bf16, float scale, float *gW, float *gb, float *sqnorm,
                      float *partial, hipStream_t stream)
{
    // 16-byte runs (8-byte for bf16) where rows and pointers allow; three
    // workgroups per CU where their smaller stage still takes chunks of four
    // or more output rows (or the whole plane)
    RowsShape s;
    const int run_bytes = 4 * (bf16 ? 2 : 4);
    const bool runs = aligned(a.X, run_bytes) && aligned(a.GY, run_bytes);
    int which = 2;
    if (runs && plan_rows(a, kSmall4, s) && (s.RC >= 4 || s.RC == s.Ho)) which = 1;
    else if (runs && plan_rows(a, kLarge4, s)) which = 0;
    else plan_rows(a, kSingle, s);
    s.vec = s.KK % 4 == 0 && aligned(gW, 16);
    const int tiles = s.ktiles * s.ctiles;
    const int direct = tiles == 1;
    float *sqout = sqnorm ? (direct ? sqnorm : partial) : nullptr;
    if (s.Cout > 32) {
        if (bf16) launch_typed<uint16_t, 2>(a, which, s, scale, gW, gb, sqout, direct, stream);
        else launch_typed<float, 2>(a, which, s, scale, gW, gb, sqout, direct, stream);
    } else {
        if (bf16) launch_typed<uint16_t, 1>(a, which, s, scale, gW, gb, sqout, direct, stream);
        else launch_typed<float, 1>(a, which, s, scale, gW, gb, sqout, direct, stream);
    }
    if (sqnorm && !direct) sum_partials(partial, a.N, tiles, sqnorm, stream);
}

}  // namespace dpg
