// Linear layer: per-sample gradients and the fused clipped sum.
//
// Per-sample gradient of y_t = W x_t + b for sample n (appendix "Vectorized
// Computation"; extra dimensions summed):
//   gW_n = s * B_n^T A_n   (d_out x d_in, K = T positions),  gb_n = s * sum_t B_n,t
// T = 1 is a rank-one outer product (linear_outer.hpp).  T > 1 is a real per-sample GEMM on
// MFMA with the squared-norm partials taken from the accumulators in the
// epilogue.
//
// Fused clipped sum: sum_n c_n gW_n = s * B^T diag(c) A, one GEMM whose K runs
// over all N*T rows, split over workgroups; partial tiles go to the workspace
// and a second kernel adds them in split order (no atomics).
#include "common.hpp"
#include "mfma_tile.hpp"
#include "linear_bf16.hpp"
#include "grad_sample_bf16.hpp"
#include "linear_outer.hpp"
#include "bf16_stage.hpp"
#include "linear_staged.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 64, kBN = 64, kBK = 32;

template <typename T>
__device__ __forceinline__ float4 load4(const T *p, i64 i);

template <>
__device__ __forceinline__ float4 load4<float>(const float *p, i64 i)
{
    return *reinterpret_cast<const float4 *>(p + i);
}

template <>
__device__ __forceinline__ float4 load4<uint16_t>(const uint16_t *p, i64 i)
{
    const uint2 u = *reinterpret_cast<const uint2 *>(p + i);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

// T = 1: the rank-one outer product (linear_outer.hpp), block = (sample, rows)
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads) void outer_kernel(const T *__restrict__ A, const T *__restrict__ B, i64 din,
                                                         i64 dout, int rows, int bps, float scale,
                                                         float *__restrict__ gW, float *__restrict__ gb,
                                                         float *__restrict__ sqnorm)
{
    louter::outer_block<T, VEC>(A, B, din, dout, rows, blockIdx.x / bps, (int)(blockIdx.x % bps), scale, gW, gb,
                                sqnorm);
}

// ---------------------------------------------------------------------------
// T > 1: per-sample GEMM on MFMA.  Block = (sample n, 64 x 64 tile of gW_n).
// MFMA rows run over j (d_in, the contiguous index of gW), so each lane ends
// with four consecutive entries of a row of gW and stores them as one float4;
// columns run over i (d_out).  Both operands are staged K-major exactly as
// they lie in memory ([t][feature]), with 16-byte loads when the rows allow;
// the next chunk of positions is loaded into registers while the current
// one is multiplied.
// ---------------------------------------------------------------------------
constexpr int kPM = 64, kPN = 64, kPK = 32;

template <typename T, int VEC>
__device__ __forceinline__ void load_group(const T *p, float (&v)[VEC])
{
    if constexpr (VEC == 4) {
        const float4 q = load4<T>(p, 0);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    } else {
        v[0] = load_elem<T>(p, 0);
    }
}

template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void ps_gemm_kernel(
    const T *__restrict__ A, const T *__restrict__ B, i64 Tn, i64 din, i64 dout, int tiles_j,
    int tiles, float scale, float *__restrict__ gW, float *__restrict__ gb,
    float *__restrict__ partial)
{
    __shared__ float As[kPK * kPM];   // [t][j]
    __shared__ float Bs[kPK * kPN];   // [t][i]
    __shared__ float red[16];
    const i64 bsw = xcd_swizzle(blockIdx.x, gridDim.x);
    const i64 n = bsw / tiles;
    const int tile = (int)(bsw % tiles);
    const int ti = tile / tiles_j, tj = tile % tiles_j;
    const i64 j0 = (i64)tj * kPM, i0 = (i64)ti * kPN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave & 1) * 32, wn = (wave >> 1) * 32;
    const T *An = A + n * Tn * din;
    const T *Bn = B + n * Tn * dout;
    const bool do_bias = gb != nullptr && tj == 0;

    // staging: VEC-wide groups, group g = tid + 256 q at row g / GPR
    constexpr int GPR = kPM / VEC;
    constexpr int NG = kPK * kPM / VEC / kThreads;
    static_assert(kPM == kPN && NG * VEC * kThreads == kPK * kPM, "staging map");
    float ra[NG][VEC], rb[NG][VEC];
    auto load = [&](i64 t0) {
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int g = tid + kThreads * q;
            const int r = g / GPR, c = (g % GPR) * VEC;
            const i64 t = t0 + r;
            const bool okA = t < Tn && j0 + c < din;   // VEC = 4: d_in % 4 == 0, whole group in or out
            const bool okB = t < Tn && i0 + c < dout;
            load_group<T, VEC>(An + (okA ? t * din + j0 + c : 0), ra[q]);
            load_group<T, VEC>(Bn + (okB ? t * dout + i0 + c : 0), rb[q]);
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                ra[q][v] = okA ? ra[q][v] : 0.0f;
                rb[q][v] = okB ? rb[q][v] : 0.0f;
            }
        }
    };
    auto store = [&]() {
#pragma unroll
        for (int q = 0; q < NG; ++q) {
            const int g = tid + kThreads * q;
            const int r = g / GPR, c = (g % GPR) * VEC;
            if constexpr (VEC == 4) {
                *reinterpret_cast<float4 *>(As + r * kPM + c) = make_float4(ra[q][0], ra[q][1], ra[q][2], ra[q][3]);
                *reinterpret_cast<float4 *>(Bs + r * kPN + c) = make_float4(rb[q][0], rb[q][1], rb[q][2], rb[q][3]);
            } else {
                As[r * kPM + c] = ra[q][0];
                Bs[r * kPN + c] = rb[q][0];
            }
        }
    };

    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
    float bias_acc = 0.0f;
    load(0);
    for (i64 t0 = 0; t0 < Tn; t0 += kPK) {
        __syncthreads();   // previous chunk consumed
        store();
        __syncthreads();
        if (t0 + kPK < Tn) load(t0 + kPK);
        const int li = lane & 31, lk = lane >> 5;
#pragma unroll
        for (int kk = 0; kk < kPK; kk += 2) {
            const float a = As[(kk + lk) * kPM + wm + li];
            const float b = Bs[(kk + lk) * kPN + wn + li];
            acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc, 0, 0, 0);
        }
        if (do_bias && tid < kPN) {
#pragma unroll 8
            for (int kk = 0; kk < kPK; ++kk) bias_acc += Bs[kk * kPN + tid];
        }
    }

    // acc[r] holds gW[i][j], j = j0 + wm + 8 (r / 4) + 4 (lane / 32) + r % 4, i = i0 + wn + lane % 32
    float sq = 0.0f;
    const i64 i = i0 + wn + (lane & 31);
    if (i < dout) {
        float *G = gW + n * dout * din + i * din;
#pragma unroll
        for (int rb4 = 0; rb4 < 4; ++rb4) {
            const i64 j = j0 + wm + 8 * rb4 + 4 * (lane >> 5);
            const float g0 = scale * acc[4 * rb4 + 0], g1 = scale * acc[4 * rb4 + 1];
            const float g2 = scale * acc[4 * rb4 + 2], g3 = scale * acc[4 * rb4 + 3];
            if (VEC == 4) {
                if (j < din) {
                    *reinterpret_cast<float4 *>(G + j) = make_float4(g0, g1, g2, g3);
                    sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
                }
            } else {
                if (j + 0 < din) { G[j + 0] = g0; sq += g0 * g0; }
                if (j + 1 < din) { G[j + 1] = g1; sq += g1 * g1; }
                if (j + 2 < din) { G[j + 2] = g2; sq += g2 * g2; }
                if (j + 3 < din) { G[j + 3] = g3; sq += g3 * g3; }
            }
        }
    }
    if (do_bias && tid < kPN && i0 + tid < dout) {
        const float g = scale * bias_acc;
        gb[n * dout + i0 + tid] = g;
        sq += g * g;
    }
    sq = block_sum(sq, red);
    if (partial && tid == 0) partial[n * tiles + tile] = sq;
}

// ---------------------------------------------------------------------------
// T > 1, fp32, staged straight into LDS (T % 16 == 0, d_in and d_out
// multiples of 4, 16-byte aligned operands).  Block = (sample n, 64 x 64
// tile of gW_n) as above.  Stages of 16 positions of both tiles (4 KB each)
// are copied by global_load_lds_dwordx4 into a ring of four, and the waves
// wait for exactly the stage they need: no operand passes through registers
// on its way to LDS, so no wait for a later stage's loads couples in.  A
// stage's operands are read into registers one stage ahead, while the
// previous stage's MFMAs run.  Inside a row the 16-byte chunks of
// odd rows are shifted by half a row, so the two rows a wave's operand read
// touches fall in different banks.  Each wave keeps two accumulators (odd
// and even k-steps: two independent MFMA chains), added at the end; the bias
// gradient is the column sum of the B operands the waves already hold.  Features past the layer's edge read a clamped valid chunk, whose
// outputs are never stored.
// ---------------------------------------------------------------------------
constexpr int kDK = 16;                          // positions per stage
constexpr int kDStages = 4;
constexpr int kDRow = kPM * 4;                   // bytes per staged row (64 floats)
constexpr int kDTile = kDK * kDRow;              // 4 KB per operand tile and stage
constexpr int kDStageBytes = 2 * kDTile;

__device__ __forceinline__ int dma_chunk_pos(int row, int chunk) { return chunk ^ (8 * (row & 1)); }

// LDS of one workgroup of the staged kernels
struct DmaShared {
    __attribute__((aligned(1024))) char ring[kDStages * kDStageBytes];
    float red[16];
    float bred[2][kPN];
};

// Tile `tile` of sample n (the body of the single-layer and grouped launches)
__device__ __forceinline__ void ps_dma_tile(const float *__restrict__ A, const float *__restrict__ B, i64 Tn,
                                            i64 din, i64 dout, int tiles_j, int tiles, i64 n, int tile,
                                            float scale, float *__restrict__ gW, float *__restrict__ gb,
                                            float *__restrict__ partial, DmaShared &sh)
{
    char *smem = sh.ring;
    float *red = sh.red;
    float (*bred)[kPN] = sh.bred;
    const int ti = tile / tiles_j, tj = tile % tiles_j;
    const i64 j0 = (i64)tj * kPM, i0 = (i64)ti * kPN;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = (wave & 1) * 32, wn = (wave >> 1) * 32;
    const bool do_bias = gb != nullptr && tj == 0;
    const int nst = (int)(Tn / kDK);
    const uint32_t lds0 = bf16s::lds_addr(smem);

    // wave w copies rows 4w .. 4w+3 of both tiles of a stage (one 1 KB
    // instruction each): lane l -> row 4w + l / 16, LDS chunk l % 16, which
    // holds feature chunk dma_chunk_pos(row, l % 16) of that row
    const int srow = 4 * wave + lane / 16;
    const int schunk = dma_chunk_pos(srow, lane % 16);
    i64 fa = j0 + 4 * schunk, fb = i0 + 4 * schunk;
    fa = fa < din ? fa : din - 4;
    fb = fb < dout ? fb : dout - 4;
    const float *An = A + n * Tn * din + (i64)srow * din + fa;
    const float *Bn = B + n * Tn * dout + (i64)srow * dout + fb;
    const uint32_t lds_a = (uint32_t)(4 * wave * kDRow), lds_b = (uint32_t)(kDTile + 4 * wave * kDRow);
    auto issue = [&](int c) {
        const uint32_t L = lds0 + (uint32_t)(c % kDStages) * kDStageBytes;
        bf16s::dma16(An + (i64)c * kDK * din, L + lds_a);
        bf16s::dma16(Bn + (i64)c * kDK * dout, L + lds_b);
    };
    constexpr int LOADS = 2;                     // per wave per stage

    f32x16 acc0, acc1;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.0f;
    // column sums of the wave's B operands: lane l holds rows of parity l / 32
    // of column wn + l % 32 (the bias gradient, from the registers the MFMAs read)
    float bias_acc = 0.0f;
    const int li = lane & 31, lk = lane >> 5;
    // operand addresses inside a stage: A feature wm + li, B feature wn + li, row kk + lk
    auto opnd = [&](int row, int f) { return row * kDRow + 16 * dma_chunk_pos(row, f >> 2) + 4 * (f & 3); };

    // a stage's operands in registers: k-steps 0, 2, .., 14 of the wave's A and B columns
    struct Ops {
        float a[kDK / 2], b[kDK / 2];
    };
    auto read_ops = [&](int c, Ops &o) {
        const char *L = smem + (c % kDStages) * kDStageBytes;
#pragma unroll
        for (int k = 0; k < kDK / 2; ++k) {
            o.a[k] = *reinterpret_cast<const float *>(L + opnd(2 * k + lk, wm + li));
            o.b[k] = *reinterpret_cast<const float *>(L + kDTile + opnd(2 * k + lk, wn + li));
        }
    };
    auto mma = [&](const Ops &o) {
#pragma unroll
        for (int k = 0; k < kDK / 2; k += 2) {
            acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(o.a[k], o.b[k], acc0, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(o.a[k + 1], o.b[k + 1], acc1, 0, 0, 0);
        }
        float s = 0.0f;
#pragma unroll
        for (int k = 0; k < kDK / 2; ++k) s += o.b[k];
        bias_acc += s;
    };
    // stage c has landed once only the loads of the `later` stages after it remain
    auto wait_landed = [&](int later) {
        if (later >= 3) bf16s::wait_vmcnt<3 * LOADS>();
        else if (later == 2) bf16s::wait_vmcnt<2 * LOADS>();
        else if (later == 1) bf16s::wait_vmcnt<LOADS>();
        else bf16s::wait_vmcnt<0>();
    };

    // Per stage c (its operands already in registers): wait for stage c+1,
    // meet at the barrier (every wave has its stage c operands, so stage c's
    // buffer may take stage c+4), issue stage c+4, then the MFMAs of stage c
    // with the reads of stage c+1 between them.
#pragma unroll
    for (int c = 0; c < kDStages; ++c)
        if (c < nst) issue(c);
    // one stage c < nst - 1: its MFMAs (operands in cur) and the reads of stage c+1 into nxt
    auto step = [&](int c, const Ops &cur, Ops &nxt) {
        wait_landed(nst - 2 - c < kDStages - 2 ? nst - 2 - c : kDStages - 2);
        bf16s::wait_lgkmcnt0();
        bf16s::stage_barrier();
        if (c + kDStages < nst) issue(c + kDStages);
        read_ops(c + 1, nxt);
        mma(cur);
#pragma unroll
        for (int k = 0; k < kDK / 2; ++k) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read (two rows)
        }
    };
    Ops x, y;   // two register sets, stages alternate between them
    if (nst > 0) {
        wait_landed(nst - 1 < kDStages - 1 ? nst - 1 : kDStages - 1);
        bf16s::stage_barrier();
        read_ops(0, x);
        int c = 0;
        for (; c + 2 < nst; c += 2) {
            step(c, x, y);
            step(c + 1, y, x);
        }
        if (c + 1 < nst) {   // two stages left
            step(c, x, y);
            x = y;
        }
        mma(x);
    }

    // acc[r] holds gW[i][j], j = j0 + wm + 8 (r / 4) + 4 (lane / 32) + r % 4, i = i0 + wn + lane % 32
    float sq = 0.0f;
    const i64 i = i0 + wn + (lane & 31);
    if (i < dout) {
        float *G = gW + n * dout * din + i * din;
#pragma unroll
        for (int rb4 = 0; rb4 < 4; ++rb4) {
            const i64 j = j0 + wm + 8 * rb4 + 4 * (lane >> 5);
            const float g0 = scale * (acc0[4 * rb4 + 0] + acc1[4 * rb4 + 0]);
            const float g1 = scale * (acc0[4 * rb4 + 1] + acc1[4 * rb4 + 1]);
            const float g2 = scale * (acc0[4 * rb4 + 2] + acc1[4 * rb4 + 2]);
            const float g3 = scale * (acc0[4 * rb4 + 3] + acc1[4 * rb4 + 3]);
            if (j < din) {   // d_in % 4 == 0: the four j are all in or all out
                *reinterpret_cast<float4 *>(G + j) = make_float4(g0, g1, g2, g3);
                sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
            }
        }
    }
    if (do_bias) {
        // waves 0 and 2 (wm == 0) hold columns 0..31 and 32..63; a column's
        // even rows (lane l) and odd rows (lane l + 32) are added in that order
        if (wm == 0 && lane < 32) bred[0][wn + lane] = bias_acc;
        if (wm == 0 && lane >= 32) bred[1][wn + lane - 32] = bias_acc;
        __syncthreads();
        if (tid < kPN && i0 + tid < dout) {
            const float g = scale * (bred[0][tid] + bred[1][tid]);
            gb[n * dout + i0 + tid] = g;
            sq += g * g;
        }
    }
    sq = block_sum(sq, red);
    if (partial && tid == 0) partial[n * tiles + tile] = sq;
}

__global__ __launch_bounds__(kThreads) void ps_gemm_dma_kernel(const float *__restrict__ A, const float *__restrict__ B,
                                                               i64 Tn, i64 din, i64 dout, int tiles_j, int tiles,
                                                               float scale, float *__restrict__ gW,
                                                               float *__restrict__ gb, float *__restrict__ partial)
{
    __shared__ DmaShared sh;
    const i64 bsw = xcd_swizzle(blockIdx.x, gridDim.x);
    ps_dma_tile(A, B, Tn, din, dout, tiles_j, tiles, bsw / tiles, (int)(bsw % tiles), scale, gW, gb, partial, sh);
}

// Several staged layers sharing N in one launch: workgroup b takes sample
// b / tiles_all and, of that sample's tiles of all layers (layer after layer),
// tile b % tiles_all, so layers that read the same B (an LSTM's two weight
// matrices) read it while it is in L2.
struct PsDmaItem {
    const float *A, *B;
    i64 T, din, dout;
    int tiles_j, tiles, tile0;
    float scale;
    float *gW, *gb, *sqnorm, *partial;
};
struct PsDmaGroup {
    int count, tiles_all;
    i64 N;
    PsDmaItem it[kPsGroupMax];
};

__global__ __launch_bounds__(kThreads) void ps_dma_group_kernel(const PsDmaGroup g)
{
    __shared__ DmaShared sh;
    const i64 bsw = xcd_swizzle(blockIdx.x, gridDim.x);
    const i64 n = bsw / g.tiles_all;
    const int r = (int)(bsw % g.tiles_all);
    int k = 0;
    while (k + 1 < g.count && g.it[k + 1].tile0 <= r) ++k;
    const PsDmaItem &L = g.it[k];
    ps_dma_tile(L.A, L.B, L.T, L.din, L.dout, L.tiles_j, L.tiles, n, r - L.tile0, L.scale, L.gW, L.gb, L.partial,
                sh);
}

// One wave per (layer, sample): sqnorm[n] = the sample's tile partials added
// as sum_partials adds them (lane l takes partials l, l+64, ..., then the
// same butterfly), so the grouped launch matches the single-layer call bit
// for bit.
__global__ __launch_bounds__(256) void ps_dma_group_sqnorm_kernel(const PsDmaGroup g)
{
    const PsDmaItem &L = g.it[blockIdx.y];
    const i64 n = (i64)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (L.sqnorm == nullptr || n >= g.N) return;
    const float *p = L.partial + n * L.tiles;
    float s = 0.0f;
    for (int t = lane; t < L.tiles; t += kWave) s += p[t];
    s = wave_sum(s);
    if (lane == 0) L.sqnorm[n] = s;
}

bool ps_dma_ok(const void *A, const void *B, const float *gW, i64 T, i64 din, i64 dout)
{
    return T >= kDK && T % kDK == 0 && din % 4 == 0 && dout % 4 == 0 && aligned(A, 16) && aligned(B, 16) &&
           aligned(gW, 16) && T * (din > dout ? din : dout) < (i64(1) << 31);
}

// ---------------------------------------------------------------------------
// Fused clipped sum: block = (split, tile).  Rows of the flattened [N*T]
// operands are scaled by s * c_n as they are staged.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void clipsum_gemm_kernel(
    const T *__restrict__ A, const T *__restrict__ B, i64 Tn, i64 rows_total, i64 rows_per_split,
    i64 din, i64 dout, int tiles_n, int tiles, float scale, const float *__restrict__ norm,
    float C, float *__restrict__ outW, float *__restrict__ outb, i64 split_strideW,
    i64 split_strideb)
{
    __shared__ float As[kBK * kBM];
    __shared__ float Bs[kBK * kBN];
    __shared__ float rs[kBK];
    const i64 bsw = xcd_swizzle(blockIdx.x, gridDim.x);
    const int split = (int)(bsw / tiles);
    const int tile = (int)(bsw % tiles);
    const int tm = tile / tiles_n, tn = tile % tiles_n;
    const i64 m0 = (i64)tm * kBM, n0 = (i64)tn * kBN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * (kBM / 2), wn = (wave & 1) * (kBN / 2);
    const i64 r0 = (i64)split * rows_per_split;
    const i64 r1 = r0 + rows_per_split < rows_total ? r0 + rows_per_split : rows_total;
    const bool do_bias = outb != nullptr && tn == 0;

    MfmaTile<kBM, kBN> t;
    t.zero();
    float bias_acc = 0.0f;

    for (i64 k0 = r0; k0 < r1; k0 += kBK) {
        if (tid < kBK) {
            const i64 k = k0 + tid;
            rs[tid] = k < r1 ? scale * clip_factor(norm[k / Tn], C) : 0.0f;
        }
        __syncthreads();
        for (int e = tid; e < kBK * kBM; e += kThreads) {
            const int kk = e / kBM, ii = e % kBM;
            const i64 k = k0 + kk, i = m0 + ii;
            As[e] = (k < r1 && i < dout) ? rs[kk] * load_elem<T>(B, k * dout + i) : 0.0f;
        }
        for (int e = tid; e < kBK * kBN; e += kThreads) {
            const int kk = e / kBN, jj = e % kBN;
            const i64 k = k0 + kk, j = n0 + jj;
            Bs[e] = (k < r1 && j < din) ? load_elem<T>(A, k * din + j) : 0.0f;
        }
        __syncthreads();
        t.template mma<kBK>(As, kBM, Bs, kBN, wm, wn, lane);
        if (do_bias && tid < kBM) {
#pragma unroll 8
            for (int kk = 0; kk < kBK; ++kk) bias_acc += As[kk * kBM + tid];
        }
        __syncthreads();
    }

    float *O = outW + (i64)split * split_strideW;
    t.for_each(wm, wn, lane, [&](int r, int c, float v) {
        const i64 i = m0 + r, j = n0 + c;
        if (i < dout && j < din) O[i * din + j] = v;
    });
    if (do_bias && tid < kBM && m0 + tid < dout) outb[(i64)split * split_strideb + m0 + tid] = bias_acc;
}

// out[e] = sum_s part[s][e], s ascending.
__global__ void split_sum_kernel(const float *__restrict__ part, int splits, i64 count,
                                 float *__restrict__ out)
{
    const i64 e = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count) return;
    float s = 0.0f;
    s = ordered_sum(part + e, count, splits);
    out[e] = s;
}

struct ClipSplit {
    int tiles_n, tiles, splits;
    i64 rows_per_split;
};

ClipSplit clip_split(i64 N, i64 T, i64 din, i64 dout)
{
    ClipSplit s;
    s.tiles_n = (int)ceil_div(din, kBN);
    s.tiles = (int)ceil_div(dout, kBM) * s.tiles_n;
    const i64 rows = N * T;
    const i64 chunks = ceil_div(rows, kBK);
    i64 want = ceil_div(1024, s.tiles);           // aim for ~1024 workgroups
    if (want > chunks) want = chunks;
    if (want > 256) want = 256;
    if (want < 1) want = 1;
    s.rows_per_split = ceil_div(chunks, want) * kBK;
    s.splits = (int)(rows > 0 ? ceil_div(rows, s.rows_per_split) : 1);
    return s;
}

}  // namespace

bool fp32_staged_ok(const void *A, const void *B, const void *gW, i64 N, i64 T, i64 din, i64 dout)
{
    return ps_dma_ok(A, B, (const float *)gW, T, din, dout) && N < (i64(1) << 40) &&
           N * ceil_div(din, kPM) * ceil_div(dout, kPN) < (i64(1) << 26);
}

int fp32_staged_parts(i64 din, i64 dout) { return (int)(ceil_div(din, kPM) * ceil_div(dout, kPN)); }

void fp32_grad_sample_group(const Fp32GroupLayer *layers, int count, i64 N, hipStream_t stream)
{
    if (count <= 0 || N <= 0) return;
    PsDmaGroup g;
    g.count = count;
    g.N = N;
    int tiles_all = 0;
    bool norms = false;
    for (int k = 0; k < count; ++k) {
        const Fp32GroupLayer &L = layers[k];
        PsDmaItem &it = g.it[k];
        it.A = (const float *)L.A;
        it.B = (const float *)L.B;
        it.T = L.T;
        it.din = L.din;
        it.dout = L.dout;
        it.tiles_j = (int)ceil_div(L.din, kPM);
        it.tiles = fp32_staged_parts(L.din, L.dout);
        it.tile0 = tiles_all;
        it.scale = L.scale;
        it.gW = L.gW;
        it.gb = L.gb;
        it.sqnorm = L.sqnorm;
        it.partial = L.sqnorm ? L.partial : nullptr;
        tiles_all += it.tiles;
        norms = norms || L.sqnorm != nullptr;
    }
    for (int k = count; k < kPsGroupMax; ++k) {
        g.it[k] = g.it[count - 1];
        g.it[k].tile0 = tiles_all;
    }
    g.tiles_all = tiles_all;
    ps_dma_group_kernel<<<(unsigned)(N * tiles_all), kThreads, 0, stream>>>(g);
    if (norms)
        ps_dma_group_sqnorm_kernel<<<dim3((unsigned)ceil_div(N, 4), (unsigned)count), 256, 0, stream>>>(g);
}

dp_status check_linear(const void *A, const void *B, dp_dtype dt, i64 N, i64 T, i64 din, i64 dout)
{
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && T >= 0 && din >= 1 && dout >= 1, DP_EINVAL);
    DPG_REQUIRE(N * T == 0 || (A != nullptr && B != nullptr), DP_EINVAL);
    DPG_REQUIRE(N < (i64(1) << 40) && T < (i64(1) << 40), DP_EINVAL);
    return DP_OK;
}

}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_grad_sample_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in,
                                                        int64_t d_out, dp_dtype dt)
{
    if (N <= 0 || T <= 1 || d_in <= 0 || d_out <= 0) return 0;
    // squared-norm partials of whichever path runs: one per 64x64 tile (fp32
    // MFMA; more than the 128x128 tiles of the bf16 kernel), or one per wave
    // and 128x128 tile (staged bf16 kernel)
    i64 parts = ceil_div(d_in, kPM) * ceil_div(d_out, kPN);
    if (dt == DP_BF16 && bf16_staged_parts(d_in, d_out) > parts) parts = bf16_staged_parts(d_in, d_out);
    return (size_t)(N * parts) * sizeof(float);
}

extern "C" dp_status dp_grad_sample_linear(const void *A, const void *B, dp_dtype dt, int64_t N,
                                           int64_t T, int64_t d_in, int64_t d_out, float scale,
                                           float *gW, float *gb, float *sqnorm, int32_t *status,
                                           void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)status;
    dp_status st = check_linear(A, B, dt, N, T, d_in, d_out);
    if (st != DP_OK) return st;
    DPG_REQUIRE(N == 0 || gW != nullptr, DP_EINVAL);
    const size_t need = dp_grad_sample_linear_workspace_bytes(N, T, d_in, d_out, dt);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) return DP_OK;

    if (T == 0) {
        // empty sum over positions: every gradient and norm is zero
        zero_fill(gW, N * d_out * d_in, stream);
        zero_fill(gb, N * d_out, stream);
        zero_fill(sqnorm, N, stream);
        return launch_status();
    }
    if (T == 1) {
        const louter::OuterPlan op = louter::outer_plan(d_in, d_out);
        const int rows = op.rows, bps = op.bps;
        const dim3 grid((unsigned)(N * bps));
        const bool vec = (d_in % 4) == 0 && aligned(A, dt == DP_F32 ? 16 : 8) && aligned(gW, 16);
        if (dt == DP_F32) {
            if (vec)
                outer_kernel<float, true><<<grid, kThreads, 0, stream>>>(
                    (const float *)A, (const float *)B, d_in, d_out, rows, bps, scale, gW, gb, sqnorm);
            else
                outer_kernel<float, false><<<grid, kThreads, 0, stream>>>(
                    (const float *)A, (const float *)B, d_in, d_out, rows, bps, scale, gW, gb, sqnorm);
        } else {
            if (vec)
                outer_kernel<uint16_t, true><<<grid, kThreads, 0, stream>>>(
                    (const uint16_t *)A, (const uint16_t *)B, d_in, d_out, rows, bps, scale, gW, gb, sqnorm);
            else
                outer_kernel<uint16_t, false><<<grid, kThreads, 0, stream>>>(
                    (const uint16_t *)A, (const uint16_t *)B, d_in, d_out, rows, bps, scale, gW, gb, sqnorm);
        }
        return launch_status();
    }

    float *partial = sqnorm ? (float *)ws : nullptr;
    if (dt == DP_BF16 && bf16_staged_ok(A, B, gW, N, T, d_in, d_out)) {
        bf16_grad_sample_staged(A, B, N, T, d_in, d_out, scale, gW, gb, partial, stream);
        if (sqnorm)
            sum_partials(partial, N, bf16_staged_parts(d_in, d_out), sqnorm, stream);
        return launch_status();
    }
    if (dt == DP_BF16 && bf16_path_ok(A, B, gW, T, d_in, d_out)) {
        bf16_grad_sample(A, B, N, T, d_in, d_out, scale, gW, gb, partial, stream);
        if (sqnorm)
            sum_partials(partial, N, bf16_tiles(d_in, d_out), sqnorm, stream);
        return launch_status();
    }
    const int tiles_j = (int)ceil_div(d_in, kPM);
    const int tiles = (int)ceil_div(d_out, kPN) * tiles_j;
    const dim3 grid((unsigned)(N * tiles));
    if (dt == DP_F32 && ps_dma_ok(A, B, gW, T, d_in, d_out)) {
        ps_gemm_dma_kernel<<<grid, kThreads, 0, stream>>>((const float *)A, (const float *)B, T, d_in, d_out,
                                                          tiles_j, tiles, scale, gW, gb, partial);
        if (sqnorm)
            sum_partials(partial, N, tiles, sqnorm, stream);
        return launch_status();
    }
    // 16-byte (fp32) / 8-byte (bf16) operand loads and float4 stores when
    // every row starts on such a boundary
    const size_t ea = dt == DP_F32 ? 16 : 8;
    const bool vec = d_in % 4 == 0 && d_out % 4 == 0 && aligned(A, ea) && aligned(B, ea) && aligned(gW, 16);
    if (dt == DP_F32) {
        if (vec)
            ps_gemm_kernel<float, 4><<<grid, kThreads, 0, stream>>>(
                (const float *)A, (const float *)B, T, d_in, d_out, tiles_j, tiles, scale, gW, gb, partial);
        else
            ps_gemm_kernel<float, 1><<<grid, kThreads, 0, stream>>>(
                (const float *)A, (const float *)B, T, d_in, d_out, tiles_j, tiles, scale, gW, gb, partial);
    } else {
        if (vec)
            ps_gemm_kernel<uint16_t, 4><<<grid, kThreads, 0, stream>>>(
                (const uint16_t *)A, (const uint16_t *)B, T, d_in, d_out, tiles_j, tiles, scale, gW, gb,
                partial);
        else
            ps_gemm_kernel<uint16_t, 1><<<grid, kThreads, 0, stream>>>(
                (const uint16_t *)A, (const uint16_t *)B, T, d_in, d_out, tiles_j, tiles, scale, gW, gb,
                partial);
    }
    if (sqnorm)
        sum_partials(partial, N, tiles, sqnorm, stream);
    return launch_status();
}

extern "C" size_t dp_clip_accumulate_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in,
                                                            int64_t d_out, dp_dtype dt)
{
    if (N <= 0 || T <= 0 || d_in <= 0 || d_out <= 0) return 0;
    const ClipSplit s = clip_split(N, T, d_in, d_out);
    size_t need = s.splits > 1 ? (size_t)s.splits * (size_t)(d_out * d_in + d_out) * sizeof(float) : 0;
    if (dt == DP_BF16) {
        const size_t b = bf16_clip_workspace(N, T, d_in, d_out);
        if (b > need) need = b;
    }
    return need;
}

extern "C" dp_status dp_clip_accumulate_linear(const void *A, const void *B, dp_dtype dt,
                                               int64_t N, int64_t T, int64_t d_in, int64_t d_out,
                                               float scale, const float *norm, float C,
                                               float *sumW, float *sumb, int32_t *status,
                                               void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)status;
    dp_status st = check_linear(A, B, dt, N, T, d_in, d_out);
    if (st != DP_OK) return st;
    DPG_REQUIRE(sumW != nullptr && (N == 0 || norm != nullptr), DP_EINVAL);
    DPG_REQUIRE(C > 0.0f, DP_EINVAL);
    const size_t need = dp_clip_accumulate_linear_workspace_bytes(N, T, d_in, d_out, dt);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N * T == 0) {
        zero_fill(sumW, d_out * d_in, stream);
        zero_fill(sumb, d_out, stream);
        return launch_status();
    }
    if (dt == DP_BF16 && bf16_path_ok(A, B, sumW, T, d_in, d_out) && (sumb == nullptr || aligned(sumb, 4))) {
        bf16_clip_accumulate(A, B, N, T, d_in, d_out, scale, norm, C, sumW, sumb, ws, stream);
        return launch_status();
    }
    const ClipSplit s = clip_split(N, T, d_in, d_out);
    const i64 cw = d_out * d_in;
    float *pw = s.splits > 1 ? (float *)ws : sumW;
    float *pb = sumb ? (s.splits > 1 ? (float *)ws + (i64)s.splits * cw : sumb) : nullptr;
    const dim3 grid((unsigned)(s.splits * s.tiles));
    if (dt == DP_F32)
        clipsum_gemm_kernel<float><<<grid, kThreads, 0, stream>>>(
            (const float *)A, (const float *)B, T, N * T, s.rows_per_split, d_in, d_out, s.tiles_n,
            s.tiles, scale, norm, C, pw, pb, cw, d_out);
    else
        clipsum_gemm_kernel<uint16_t><<<grid, kThreads, 0, stream>>>(
            (const uint16_t *)A, (const uint16_t *)B, T, N * T, s.rows_per_split, d_in, d_out,
            s.tiles_n, s.tiles, scale, norm, C, pw, pb, cw, d_out);
    if (s.splits > 1) {
        split_sum_kernel<<<(unsigned)ceil_div(cw, 256), 256, 0, stream>>>(pw, s.splits, cw, sumW);
        if (sumb)
            split_sum_kernel<<<(unsigned)ceil_div(d_out, 256), 256, 0, stream>>>(pb, s.splits, d_out, sumb);
    }
    return launch_status();
}
