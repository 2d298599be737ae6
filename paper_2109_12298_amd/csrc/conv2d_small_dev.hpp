// Device side of the one-workgroup-per-sample Conv2d per-sample gradients:
// the shape record, the per-sample body (shared by the single-layer kernel
// and the grouped per-sample-gradient kernel) and its host-side planning.
#pragma once

#include <type_traits>

#include "bf16_stage.hpp"
#include "common.hpp"
#include "conv2d_small.hpp"

namespace dpg {
namespace csmall {

typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kSmallLds = 48 * 1024;      // bytes of dynamic LDS
constexpr int kBatch = 16;                // global loads in flight per thread per round

struct SmallShape {
    int Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
    int Hp, Wp, plane, L, Lp, KK, khw;
    int gst;                      // row stride of the staged backprop (see make_small)
    int nbm, nbn;                 // 16-blocks over kk and co
    int bpw;                      // blocks per wave: 1, 2, 4 or 8
    int gs_off, po_off;           // LDS float offsets of the backprop and the position table
    int ko_off, bp_off;           // ... of the weight-column offset table and the bias partials
    int vec;                      // float4 stores of gW
    int xplain, gplain;           // input planes (unpadded) / backprop rows kept as they lie in memory
    int xdma, gdma;               // ... and staged by direct-to-LDS copies (fp32, 16-byte aligned)
    float inv_hw, inv_w, inv_l, inv_wo, inv_khw, inv_kw;
    // stepping a thread's element index by kThreads: the input's (row, column)
    // advance and LDS slot advance, and the backprop's position and slot advance
    int xd_w, xd_h, xd_slot, gd_p, gd_slot;
};

constexpr int kMaxBpw = 8;        // accumulator blocks a wave holds at once

// q = x / d, r = x % d for 0 <= x < 2^22 through a float reciprocal, corrected
// to the exact quotient (the estimate is off by at most one)
__device__ __forceinline__ void fdivmod(int x, int d, float inv_d, int &q, int &r)
{
    q = (int)((float)x * inv_d);
    r = x - q * d;
    q += (r >= d ? 1 : 0) - (r < 0 ? 1 : 0);
    r = x - q * d;
}

// U position steps (4 positions each: lane group kq takes position p0 + 4u + kq)
// of a wave's BPW blocks: every LDS read first, then the MFMAs
template <int BPW, int U, bool MASK>
__device__ __forceinline__ void contract_step(const float *Xs, const float *Gs, const int *Po, const int (&koff)[BPW],
                                              const int (&goff)[BPW], int p0, int kq, int L, f32x4_t (&acc)[BPW])
{
    int po[U];
#pragma unroll
    for (int u = 0; u < U; ++u) po[u] = Po[p0 + 4 * u + kq];
    float a[U][BPW], b[U][BPW];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < BPW; ++j) {
            a[u][j] = Xs[koff[j] + po[u]];
            b[u][j] = Gs[goff[j] + p0 + 4 * u];
        }
    if (MASK) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const bool in = p0 + 4 * u + kq < L;
#pragma unroll
            for (int j = 0; j < BPW; ++j) {
                a[u][j] = in ? a[u][j] : 0.0f;
                b[u][j] = in ? b[u][j] : 0.0f;
            }
        }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int j = 0; j < BPW; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u][j], b[u][j], acc[j], 0, 0, 0);
}

// Sample n's gradients by one workgroup of kThreads threads; `lds` holds
// lds_floats(s) floats of dynamic LDS, 16-byte aligned.
template <typename T, int BPW>
__device__ __forceinline__ void conv_small_sample(const T *__restrict__ X, const T *__restrict__ GY, const SmallShape &s,
                                                  float scale, float *__restrict__ gW, float *__restrict__ gb,
                                                  float *__restrict__ sqnorm, i64 n, float *lds)
{
    __shared__ float red[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    float *Xs = lds;                             // [Cin][Hp][Wp], zero halo
    float *Gs = lds + s.gs_off;                  // [Cout][gst], positions 0 .. L-1 used
    int *Po = reinterpret_cast<int *>(lds + s.po_off);   // [Lp]
    int *Ko = reinterpret_cast<int *>(lds + s.ko_off);   // [KK]: plane offset of weight column kk
    const T *Xn = X + n * s.Cin * s.H * s.W;
    const T *Gn = GY + n * s.Cout * s.L;
    const int xcount = s.Cin * s.H * s.W, gcount = s.Cout * s.L;

    // ---- staging: clear the planes and build the position table while the
    // first round of loads is in flight, then write the loaded values.  A
    // thread's elements are tid, tid + kThreads, ...; their LDS slots are
    // stepped incrementally (one division per thread, not per element).
    int xw, xh, xslot, gp, gslot;
    {
        int c, r, co;
        fdivmod(tid, s.H * s.W, s.inv_hw, c, r);
        fdivmod(r, s.W, s.inv_w, xh, xw);
        xslot = c * s.plane + (xh + s.ph) * s.Wp + xw + s.pw;
        fdivmod(tid, s.L, s.inv_l, co, gp);
        gslot = co * s.gst + gp;
    }
    const T *xp = Xn + tid;
    const T *gp_ = Gn + tid;
    // A tensor kept in its own layout (fp32, 16-byte aligned, a multiple of
    // four elements; the input also unpadded) is copied into LDS by
    // global_load_lds_dwordx4: 1 KB per wave instruction, no VGPR round trip,
    // no per-element index work.  Lanes past its end re-read its first chunk
    // into the slack that follows it in LDS.  The other tensor goes through
    // registers below.
    bool xdma = false, gdma = false;
    if constexpr (std::is_same<T, float>::value) {
        xdma = s.xdma != 0;
        gdma = s.gdma != 0;
        const int nx = xdma ? xcount / 4 : 0, ng = gdma ? gcount / 4 : 0;
        const int ix = (nx + 63) / 64, ig = (ng + 63) / 64;
        const uint32_t lx = bf16s::lds_addr(Xs), lg = bf16s::lds_addr(Gs);
        for (int i = wave; i < ix + ig; i += kWaves) {
            if (i < ix) {
                const int c = i * 64 + lane;
                bf16s::dma16(Xn + 4 * (c < nx ? c : 0), lx + (uint32_t)i * 1024u);
            } else {
                const int c = (i - ix) * 64 + lane;
                bf16s::dma16(Gn + 4 * (c < ng ? c : 0), lg + (uint32_t)(i - ix) * 1024u);
            }
        }
    }
    // The register path: rounds of kThreads elements, up to the larger of
    // the two counts it handles (a wave-uniform test, so unused rounds cost
    // no vector instructions).  The halo is cleared and the position and
    // weight-column tables are built while the first round's loads (and the
    // copies above) are in flight.
    const int xreg = xdma ? 0 : xcount, greg = gdma ? 0 : gcount;
    const int lim = xreg > greg ? xreg : greg;
    for (int e0 = 0; e0 == 0 || e0 < lim; e0 += kBatch * kThreads) {
        float xv[kBatch], gv[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            if (e0 + j * kThreads >= lim) break;
            const int e = e0 + j * kThreads + tid;
            xv[j] = e < xreg ? load_elem<T>(xp, e0 + j * kThreads) : 0.0f;
            gv[j] = e < greg ? load_elem<T>(gp_, e0 + j * kThreads) : 0.0f;
        }
        if (e0 == 0) {
            if (!xdma)
                for (int i = tid; i < s.Cin * s.plane; i += kThreads) Xs[i] = 0.0f;
            for (int p = tid; p < s.Lp; p += kThreads) {
                int oh, ow;
                fdivmod(p, s.Wo, s.inv_wo, oh, ow);
                Po[p] = p < s.L ? oh * s.sh * s.Wp + ow * s.sw : 0;
            }
            for (int k = tid; k < s.KK; k += kThreads) {
                int ci, rem, u, v;
                fdivmod(k, s.khw, s.inv_khw, ci, rem);
                fdivmod(rem, s.kw, s.inv_kw, u, v);
                Ko[k] = ci * s.plane + u * s.Wp + v;
            }
            __syncthreads();   // the cleared halo is in place before the interior lands
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
            if (e0 + j * kThreads >= lim) break;
            const int e = e0 + j * kThreads + tid;
            if (e < xreg) Xs[xslot] = xv[j];
            if (e < greg) Gs[gslot] = gv[j];
            // element e + kThreads: column carry into the row, row carry into the plane
            xw += s.xd_w;
            xslot += s.xd_slot;
            if (xw >= s.W) {
                xw -= s.W;
                xslot += s.Wp - s.W;
                ++xh;
            }
            xh += s.xd_h;
            if (xh >= s.H) {
                xh -= s.H;
                xslot += s.plane - s.H * s.Wp;
            }
            gp += s.gd_p;
            gslot += s.gd_slot;
            if (gp >= s.L) {
                gp -= s.L;
                gslot += s.gst - s.L;
            }
        }
    }
    if (xdma || gdma) bf16s::wait_vmcnt<0>();
    __syncthreads();

    // ---- bias: thread (seg, co) adds positions seg, seg + segs, ...; the
    // segments are then added in order
    float sq = 0.0f;
    if (gb != nullptr) {
        float *bpart = lds + s.bp_off;    // [segs][Cout]
        const int segs = kThreads / s.Cout;
        const int co = tid % s.Cout, seg = tid / s.Cout;
        if (seg < segs) {
            float b = 0.0f;
            for (int p = seg; p < s.L; p += segs) b += Gs[co * s.gst + p];
            bpart[seg * s.Cout + co] = b;
        }
        __syncthreads();
        if (tid < s.Cout) {
            float b = 0.0f;
            for (int k = 0; k < segs; ++k) b += bpart[k * s.Cout + tid];
            b *= scale;
            gb[n * s.Cout + tid] = b;
            sq += b * b;
        }
    }

    // ---- the contraction.  Wave w owns blocks w*BPW .. w*BPW + BPW - 1 in
    // co-major order (so its blocks mostly share one co range, whose backprop
    // reads then serve them all) and holds all their accumulators at once.
    // Lanes of a kk or co past the end read a valid address (kk 0, co 0):
    // they feed only output rows and columns that are never stored.
    const int nblocks = s.nbm * s.nbn;
    const int r16 = lane & 15, kq = lane >> 4;
    float *G = gW + n * s.Cout * s.KK;
    const int b0 = __builtin_amdgcn_readfirstlane(wave) * BPW;
    // the wave's blocks (bm, bn) in order, stepped from the first one
    int bms[BPW], bns[BPW];
    {
        int bm = b0 % s.nbm, bn = b0 / s.nbm;
#pragma unroll
        for (int j = 0; j < BPW; ++j) {
            bms[j] = bm;
            bns[j] = bn;
            if (++bm == s.nbm) {
                bm = 0;
                ++bn;
            }
        }
    }
    int koff[BPW], goff[BPW];
    f32x4_t acc[BPW];
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
        const bool live = b0 + j < nblocks;
        const int kk = bms[j] * 16 + r16;
        koff[j] = Ko[live && kk < s.KK ? kk : 0];
        const int co = bns[j] * 16 + r16;
        goff[j] = (live && co < s.Cout ? co : 0) * s.gst + kq;
        acc[j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    }
    // U position steps per iteration, so that the table reads and the
    // operand reads that depend on them are in flight together; the chunk
    // that holds the end of the positions masks what lies past it
    constexpr int U = BPW >= 8 ? 1 : 8 / BPW;
    const int Lfull = s.L - s.L % (4 * U);
    for (int p0 = 0; p0 < Lfull; p0 += 4 * U) contract_step<BPW, U, false>(Xs, Gs, Po, koff, goff, p0, kq, s.L, acc);
    if (Lfull < s.L) contract_step<BPW, U, true>(Xs, Gs, Po, koff, goff, Lfull, kq, s.L, acc);
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
        if (b0 + j >= nblocks) continue;
        const int bm = bms[j], bn = bns[j];
        const int co = bn * 16 + r16;
        // lane holds kk = bm*16 + 4*kq + r (r = 0..3) of column co
        const int kk0 = bm * 16 + 4 * kq;
        if (co < s.Cout) {
            const float g0 = scale * acc[j][0], g1 = scale * acc[j][1];
            const float g2 = scale * acc[j][2], g3 = scale * acc[j][3];
            float *dst = G + (i64)co * s.KK + kk0;
            if (s.vec && kk0 + 3 < s.KK) {
                store_stream4(dst, g0, g1, g2, g3);
                sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
            } else {
                if (kk0 + 0 < s.KK) { dst[0] = g0; sq += g0 * g0; }
                if (kk0 + 1 < s.KK) { dst[1] = g1; sq += g1 * g1; }
                if (kk0 + 2 < s.KK) { dst[2] = g2; sq += g2 * g2; }
                if (kk0 + 3 < s.KK) { dst[3] = g3; sq += g3 * g3; }
            }
        }
    }

    // ---- the sample's squared norm: waves' sums in wave order
    sq = wave_sum(sq);
    if (lane == 0) red[wave] = sq;
    __syncthreads();
    if (tid == 0 && sqnorm) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += red[w];
        sqnorm[n] = t;
    }
}

// floats of dynamic LDS a workgroup needs
inline long lds_floats(const SmallShape &s)
{
    // the bias partials [segs][Cout] follow the weight-column table
    return (long)s.bp_off + kThreads;
}

// the shape's derived sizes; false if the sample does not fit
inline bool make_small(const ConvSmallArgs &a, SmallShape &s)
{
    s.Cin = (int)a.Cin; s.H = (int)a.H; s.W = (int)a.W; s.Cout = (int)a.Cout;
    s.kh = (int)a.kh; s.kw = (int)a.kw; s.sh = (int)a.sh; s.sw = (int)a.sw; s.ph = (int)a.ph; s.pw = (int)a.pw;
    s.Ho = (int)a.Ho; s.Wo = (int)a.Wo;
    s.Hp = s.H + 2 * s.ph;
    s.Wp = s.W + 2 * s.pw;
    s.plane = s.Hp * s.Wp;
    s.L = s.Ho * s.Wo;
    s.Lp = (s.L + 31) & ~31;
    s.khw = s.kh * s.kw;
    s.KK = s.Cin * s.khw;
    s.nbm = (s.KK + 15) / 16;
    s.nbn = (s.Cout + 15) / 16;
    s.bpw = 1;
    while (s.bpw * kWaves < s.nbm * s.nbn) s.bpw *= 2;
    // A tensor whose element count is a multiple of four (and, for the
    // input, without padding) keeps its own layout in LDS (backprop rows of
    // L positions), followed by slack for the direct copies' last wave
    // instruction (whole 1 KB blocks) and, for the backprop, for the masked
    // final step's reads past the last row.  Otherwise a backprop row is
    // padded to 4 x odd floats, so that the 16 rows x 4 positions a wave reads
    // at once fall in 64 different banks (L = 4 x odd, like the MNIST conv1's
    // 196, has that property unpadded).
    s.xplain = s.ph == 0 && s.pw == 0 && (s.Cin * s.H * s.W) % 4 == 0;
    s.gplain = (s.Cout * s.L) % 4 == 0;
    s.xdma = s.gdma = 0;
    // (direct copies write 16-byte-aligned LDS, so a region they fill starts
    // on a 256-byte boundary)
    s.gs_off = (s.xplain || s.gplain) ? (s.Cin * s.plane + 63) & ~63 : s.Cin * s.plane;
    if (s.xplain) s.gs_off = (s.Cin * s.plane + 255) & ~255;
    if (s.gplain) {
        s.gst = s.L;
        s.po_off = s.gs_off + ((s.Cout * s.L + 32 + 255) & ~255);
    } else {
        s.gst = s.Lp + 4;
        s.po_off = s.gs_off + s.Cout * s.gst;
    }
    s.ko_off = s.po_off + s.Lp;
    s.bp_off = s.ko_off + s.KK;
    s.inv_hw = 1.0f / (float)(s.H * s.W);
    s.inv_w = 1.0f / (float)s.W;
    s.inv_l = 1.0f / (float)s.L;
    s.inv_wo = 1.0f / (float)s.Wo;
    s.inv_khw = 1.0f / (float)s.khw;
    s.inv_kw = 1.0f / (float)s.kw;
    {
        const int rows = kThreads / s.W;
        s.xd_w = kThreads % s.W;
        s.xd_h = rows % s.H;
        s.xd_slot = (rows / s.H) * s.plane + s.xd_h * s.Wp + s.xd_w;
        s.gd_p = kThreads % s.L;
        s.gd_slot = (kThreads / s.L) * s.gst + s.gd_p;
    }
    s.vec = 0;
    return a.Cout <= kThreads && lds_floats(s) * 4 <= kSmallLds && s.bpw <= kMaxBpw &&
           (long)s.Cin * s.H * s.W < (1L << 22) && (long)s.Cout * s.L < (1L << 22);
}

}  // namespace csmall
}  // namespace dpg
