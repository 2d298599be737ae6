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
// gradient, and writes one float per sample instead of d_out * d_in.  The
// flops per byte read are T / 2 (bf16), so at transformer shapes the call is
// bound by reading A and B once.
//
// Work unit: (layer, sample, 64 x 64 tile pair (bi <= bj) of the Grams,
// feature chunk).  A workgroup of four waves walks the features of A, then
// those of B, in stages of 128 bytes per position row (64 bf16 or 32 fp32
// features) of the tile's i-block rows and j-block rows (one block when bi =
// bj): the stages are copied straight into LDS by 16-byte direct loads,
// several stages in flight, each row's 16-byte chunks swizzled so that the
// operand reads (one chunk from each of 32 rows) are free of bank conflicts.
// Both Grams contract over the feature index, the contiguous one in memory,
// so an MFMA operand is one 16-byte chunk of one row: eight bf16 features
// for v_mfma_f32_32x32x16_bf16, or four fp32 features for four
// v_mfma_f32_32x32x2f32 (the order in which features are contracted is
// immaterial as long as both operands share it).  The four waves split each
// stage's k-steps and each computes the whole pair, so every operand
// fragment read from LDS feeds two MFMAs; LDS bandwidth, not the MFMAs,
// bounds the loop.  Rows past T and features past d read as zeros.
//
// With one chunk (a launch with enough units to fill the GPU: the usual case
// once the layers of a step share the launch) the workgroup ends with G_A's
// and G_B's tiles (its waves' shares added through LDS), so it forms
// sum G_B (G_A + bias) itself, counts an off-diagonal pair twice (the Grams are symmetric) and
// writes s^2 times that: nothing is written but one float per (sample,
// pair).  With several chunks (a small batch) each chunk writes its two
// partial tiles and a second launch adds them in chunk order before forming
// the product.  The pairs of a sample are then added in pair order.
//
// The units of a launch are all its layers' (a grouped call): a layer's
// workgroups are numbered so that the pairs and chunks of one sample run on
// one XCD at once (workgroups are dealt to the eight XCDs in turn), where
// the pairs that share row blocks read them from that XCD's L2; layers with
// more features per sample come first.
#include "bf16_stage.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kBT = 64;                               // Gram tile edge (positions)
constexpr int kRowBytes = 128;                        // bytes of one position row per stage
constexpr int kStageBytes = 2 * kBT * kRowBytes;      // the i-block's rows, then the j-block's
#ifndef DPG_GHOST_STAGES
#define DPG_GHOST_STAGES 4
#endif
constexpr int kStages = DPG_GHOST_STAGES;             // stages in the LDS ring (64 KB at 4)
constexpr int kGroupMax = 16;                         // layers per launch table
constexpr int kFill = 512;                            // workgroups that give every CU two
constexpr int kTile = kBT * kBT;                      // floats of one partial Gram tile

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// the source of every 16-byte chunk that lies past T or past d (never written)
__device__ __attribute__((aligned(64))) uint32_t g_ghost_zero[16];

// One layer of a launch.  out[n * pairs + p] receives the value of (sample n,
// pair p): part when pairs > 1 (then added into sqnorm by the pair sum),
// else sqnorm itself.
struct GhostLayer {
    const void *A, *B;
    float *out, *tiles, *part, *sqnorm;
    i64 T, din, dout;
    int nb, pairs, chunks, sa, sb;   // row blocks, tile pairs, feature chunks, stages over d_in and d_out
    int blk0, cblk0;                 // first workgroup of the layer in the Gram and the combine launches
    float bias, s2;
};

struct GhostGroup {
    i64 N;
    int count;
    GhostLayer L[kGroupMax];
};

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

// the layer of workgroup b: the last whose first workgroup is at or before b
__device__ __forceinline__ int layer_of(const GhostGroup &g, int b, bool combine)
{
    int k = 0;
    while (k + 1 < g.count && (combine ? g.L[k + 1].cblk0 : g.L[k + 1].blk0) <= b) ++k;
    return k;
}

// s_waitcnt vmcnt(later * LOADS) for a run-time later in [0, MAXL]
template <int LOADS, int MAXL>
__device__ __forceinline__ void wait_later(int later)
{
    if constexpr (MAXL == 0) {
        bf16s::wait_vmcnt<0>();
    } else {
        if (later >= MAXL) bf16s::wait_vmcnt<MAXL * LOADS>();
        else wait_later<LOADS, MAXL - 1>(later);
    }
}

// Chunk q of staged row r sits at chunk position q ^ swz(r).  Rows are 128
// bytes, so two rows span the 256 bytes of the LDS banks; an operand read
// takes one chunk from each of 32 consecutive rows, and with this swizzle any
// 16 consecutive rows put that chunk in 16 different 16-byte bank groups.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

__device__ __forceinline__ uint32_t elem_bits(uint16_t v) { return v; }
__device__ __forceinline__ uint32_t elem_bits(float v) { return __float_as_uint(v); }

__device__ __forceinline__ void mma_chunk(const uint4 &a, const uint4 &b, f32x16_t &acc, uint16_t)
{
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b),
                                                  acc, 0, 0, 0);
}

__device__ __forceinline__ void mma_chunk(const uint4 &a, const uint4 &b, f32x16_t &acc, float)
{
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
}

// Weight of 32 x 32 block b = 2 x + y of a pair's tiles in the pair's value:
// a diagonal pair (bi = bj) leaves out block (1, 0), the transpose of (0, 1)
// (both Grams are symmetric), and counts (0, 1) twice.
__host__ __device__ __forceinline__ float block_weight(int b, bool diag)
{
    return diag ? (b == 1 ? 2.0f : b == 2 ? 0.0f : 1.0f) : 1.0f;
}

// One work unit: sample n, pair p = (bi, bj), chunk c of layer L.  VEC:
// every row is 16-byte aligned and d_in, d_out are whole chunks, so the
// stages are direct loads; otherwise each thread loads its chunks element by
// element (bounds-checked) and stores them to LDS itself.
//
// Wave w = 2 kh + x computes the blocks (x, 0) and (x, 1) of the pair (x
// over the i-block's halves, y over the j-block's) over k-steps kh and kh + 2
// of every stage (16-byte chunks 2 s and 2 s + 1 of each row for k-step s:
// lanes 0-31 the first, 32-63 the second).  Per k-step it reads the i-half
// and both j-halves (a diagonal pair: the two halves, the i-half being one
// of them) for two MFMAs, and a stage's reads are issued while the MFMAs of
// the stage before run.  At the end the two k-parities' tiles are added
// through LDS (kh = 0 first).
template <typename T, bool VEC, bool DIAG>
__device__ __forceinline__ void gram_unit(const GhostLayer &L, i64 n, int p, int bi, int bj, int c, char *smem,
                                          float *red)
{
    constexpr int EPC = 16 / (int)sizeof(T);                 // elements per 16-byte chunk
    constexpr int F = kRowBytes / (int)sizeof(T);            // features per stage
    constexpr int ROWS = DIAG ? kBT : 2 * kBT;               // staged rows
    constexpr int LOADS = ROWS * kRowBytes / 1024 / kWaves;  // 16-byte loads per lane per stage
    static_assert(kStages * kStageBytes >= 2 * kTile * (int)sizeof(float), "the final sum reuses the ring");
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int x = wave & 1, kh = wave >> 1;
    const i64 Tn = L.T, din = L.din, dout = L.dout;
    const int C = L.chunks;
    const int a0 = (int)((i64)c * L.sa / C), a1 = (int)((i64)(c + 1) * L.sa / C);
    const int b0 = (int)((i64)c * L.sb / C), b1 = (int)((i64)(c + 1) * L.sb / C);
    const int na = a1 - a0, nst = na + (b1 - b0);
    const T *An = reinterpret_cast<const T *>(L.A) + n * Tn * din;
    const T *Bn = reinterpret_cast<const T *>(L.B) + n * Tn * dout;

    // this lane's share of a stage: load r covers LDS bytes 1024 a + 16 lane,
    // a = wave + 4 r, i.e. staged row 8 a + lane / 8, chunk position lane % 8
    // (which holds chunk (lane % 8) ^ swz(row))
    int trow[LOADS];
    uint32_t fq[LOADS];
#pragma unroll
    for (int r = 0; r < LOADS; ++r) {
        const int a = wave + kWaves * r;
        const int row = 8 * a + (lane >> 3);
        const int q = (lane & 7) ^ swz(row);
        const i64 t = row < kBT ? (i64)bi * kBT + row : (i64)bj * kBT + (row - kBT);
        // a row past T never passes the feature test below
        fq[r] = t < Tn ? (uint32_t)(q * EPC) : 0x80000000u;
        trow[r] = t < Tn ? (int)t : 0;
    }
    const uint32_t lds0 = bf16s::lds_addr(smem);
    // the zero source's address, held in registers (not reloaded per stage)
    uint64_t zaddr = reinterpret_cast<uint64_t>(g_ghost_zero);
    asm volatile("" : "+s"(zaddr));
    const void *zero = reinterpret_cast<const void *>(zaddr);
    auto issue = [&](int k, int slot) {
        const bool onA = k < na;
        const int f0 = (onA ? a0 + k : b0 + (k - na)) * F;
        const uint32_t d = (uint32_t)(onA ? din : dout);
        const T *X = onA ? An : Bn;
#pragma unroll
        for (int r = 0; r < LOADS; ++r) {
            const int a = wave + kWaves * r;
            const uint32_t f = (uint32_t)f0 + fq[r];        // f0 < 2^31: no wrap
            const int off = trow[r] * (int)d + (int)f;
            if constexpr (VEC) {
                const void *src = f < d ? (const void *)(X + off) : zero;
                bf16s::dma16(src, lds0 + (uint32_t)(slot * kStageBytes + a * 1024));
            } else {
                uint32_t wd[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) wd[e] = 0u;
#pragma unroll
                for (int e = 0; e < EPC; ++e) {
                    const uint32_t v = f + (uint32_t)e < d ? elem_bits(X[off + e]) : 0u;
                    wd[e * (int)sizeof(T) / 4] |= v << (8 * ((e * (int)sizeof(T)) & 3));
                }
                *reinterpret_cast<uint4 *>(smem + slot * kStageBytes + a * 1024 + 16 * lane) =
                    make_uint4(wd[0], wd[1], wd[2], wd[3]);
            }
        }
    };

    // LDS offsets of the wave's fragments in k-step s = kh + 2 u: the j-halves
    // (rows 32 y + lane % 32 of the j-block) and, off the diagonal, the i-half
    constexpr int NF = DIAG ? 2 : 3;
    int of[2][NF];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        const int ch = 2 * (kh + 2 * u) + (lane >> 5);
#pragma unroll
        for (int f = 0; f < NF; ++f) {
            const int row = f < 2 ? (DIAG ? 0 : kBT) + 32 * f + (lane & 31) : 32 * x + (lane & 31);
            of[u][f] = row * kRowBytes + 16 * (ch ^ swz(row));
        }
    }
    struct Frags {
        uint4 v[2][NF];
    };
    auto read = [&](int slot, Frags &fr) {
        const char *Ls = smem + slot * kStageBytes;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int f = 0; f < NF; ++f) fr.v[u][f] = *reinterpret_cast<const uint4 *>(Ls + of[u][f]);
    };

    f32x16_t acc[2], accA[2];     // blocks (x, 0), (x, 1) of G_B and of G_A
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[y][r] = accA[y][r] = 0.0f;
    auto mma = [&](const Frags &fr, f32x16_t (&G)[2]) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const uint4 &j0 = fr.v[u][0], &j1 = fr.v[u][1];
            uint4 i;
            if constexpr (DIAG) {
                i = x ? j1 : j0;
            } else {
                i = fr.v[u][NF - 1];
            }
            mma_chunk(i, j0, G[0], T());
            mma_chunk(i, j1, G[1], T());
        }
    };

#pragma unroll
    for (int k = 0; k < kStages - 1; ++k)
        if (k < nst) issue(k, k);
    // stage k: wait for its loads, then (all waves) for everyone's; refill the
    // slot of stage k - 1, whose reads every wave has finished
    auto arrive = [&](int k) {
        if constexpr (VEC) {
            const int later = nst - 1 - k < kStages - 2 ? nst - 1 - k : kStages - 2;
            wait_later<LOADS, kStages - 2>(later);
        }
        bf16s::wait_lgkmcnt0();
        bf16s::stage_barrier();
        if (k + kStages - 1 < nst) issue(k + kStages - 1, (k + kStages - 1) % kStages);
    };
    // stages k0 .. k1 - 1 into G: iteration k reads stage k into nxt while the
    // MFMAs of stage k - 1 run on cur.  The A side and the B side are two such
    // loops, each with its own accumulators (the loads run on across them).
    auto run = [&](int k0, int k1, f32x16_t (&G)[2]) {
        if (k0 >= k1) return;
        Frags fx, fy;
        arrive(k0);
        read(k0 % kStages, fx);
        int k = k0 + 1;
        for (; k + 1 < k1; k += 2) {
            arrive(k);
            read(k % kStages, fy);
            mma(fx, G);
            arrive(k + 1);
            read((k + 1) % kStages, fx);
            mma(fy, G);
        }
        if (k < k1) {
            arrive(k);
            read(k % kStages, fy);
            mma(fx, G);
            fx = fy;
        }
        mma(fx, G);
    };
    run(0, na, accA);
    run(na, nst, acc);

    // the two k-parities' blocks added (kh = 0 first), G_A then G_B, through
    // two 16 KB regions of the ring: register group q (registers 4 q .. 4 q +
    // 3) of lane l of block b sits at float 4 ((4 b + q) 64 + l), so a wave's
    // 16-byte stores and loads are consecutive.  Thread t ends with entries
    // 16 t .. 16 t + 15 (block t / 64, lane t % 64, registers 0-15).
    float ga[16], gb[16];
    float *R = reinterpret_cast<float *>(smem);
    auto add_parities = [&](const f32x16_t (&v)[2], float (&out)[16]) {
        __syncthreads();                  // the ring (or the last sum) is free
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                *reinterpret_cast<float4 *>(R + kh * kTile + 4 * ((4 * (2 * x + y) + q) * 64 + lane)) =
                    make_float4(v[y][4 * q], v[y][4 * q + 1], v[y][4 * q + 2], v[y][4 * q + 3]);
        __syncthreads();
        const int b = tid >> 6;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 e = *reinterpret_cast<const float4 *>(R + 4 * ((4 * b + q) * 64 + lane));
            const float4 g = *reinterpret_cast<const float4 *>(R + kTile + 4 * ((4 * b + q) * 64 + lane));
            out[4 * q] = e.x + g.x; out[4 * q + 1] = e.y + g.y; out[4 * q + 2] = e.z + g.z; out[4 * q + 3] = e.w + g.w;
        }
    };
    add_parities(accA, ga);
    add_parities(acc, gb);

    if (C == 1) {
        float s = 0.0f;
#pragma unroll
        for (int r = 0; r < 16; ++r) s += gb[r] * (ga[r] + L.bias);
        s = wave_sum(s * block_weight(tid >> 6, DIAG));
        if (lane == 0) red[wave] = s;
        __syncthreads();
        if (tid == 0) {
            float t = 0.0f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) t += red[w];
            L.out[n * L.pairs + p] = L.s2 * (DIAG ? t : 2.0f * t);
        }
    } else {
        // the two partial tiles, thread t's 16 entries at 16 t
        float *tA = L.tiles + ((size_t)((n * L.pairs + p) * C + c) * 2) * kTile + tid * 16;
        float4 *oA = reinterpret_cast<float4 *>(tA);
        float4 *oB = reinterpret_cast<float4 *>(tA + kTile);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            oA[q] = make_float4(ga[4 * q], ga[4 * q + 1], ga[4 * q + 2], ga[4 * q + 3]);
            oB[q] = make_float4(gb[4 * q], gb[4 * q + 1], gb[4 * q + 2], gb[4 * q + 3]);
        }
    }
}

// Workgroup b of layer k (local index l = b - blk0): XCD x = l % 8 takes,
// in turn, the pairs * chunks workgroups of samples x, x + 8, ...
template <typename T, bool VEC>
__global__ __launch_bounds__(kThreads, 2) void ghost_gram_kernel(const GhostGroup g)
{
    __shared__ __attribute__((aligned(1024))) char smem[kStages * kStageBytes];
    __shared__ float red[kWaves];
    const int b = (int)blockIdx.x;
    const GhostLayer &L = g.L[layer_of(g, b, false)];
    const int l = b - L.blk0;
    const int m = L.pairs * L.chunks;
    const int kk = l >> 3;
    const i64 n = 8 * (i64)(kk / m) + (l & 7);
    if (n >= g.N) return;
    const int j = kk % m;
    const int p = j / L.chunks, c = j % L.chunks;
    int bi, bj;
    pair_of(p, L.nb, bi, bj);
    if (bi == bj) gram_unit<T, VEC, true>(L, n, p, bi, bj, c, smem, red);
    else gram_unit<T, VEC, false>(L, n, p, bi, bj, c, smem, red);
}

// Several chunks: one workgroup per (layer, sample, pair); thread i owns
// entries 16 i .. 16 i + 15 of the two tiles, adds the chunks in chunk order
// and forms the pair's value as the one-chunk path does.
__global__ __launch_bounds__(kThreads) void ghost_combine_kernel(const GhostGroup g)
{
    __shared__ float red[kWaves];
    const int b = (int)blockIdx.x;
    const GhostLayer &L = g.L[layer_of(g, b, true)];
    const int u = b - L.cblk0;
    const i64 n = u / L.pairs;
    const int p = u % L.pairs;
    int bi, bj;
    pair_of(p, L.nb, bi, bj);
    const float *base = L.tiles + (size_t)(n * L.pairs + p) * L.chunks * 2 * kTile + threadIdx.x * 16;
    float ga[16], gb[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) ga[r] = gb[r] = 0.0f;
    for (int c = 0; c < L.chunks; ++c) {
        const float4 *ta = reinterpret_cast<const float4 *>(base + (size_t)(2 * c) * kTile);
        const float4 *tb = reinterpret_cast<const float4 *>(base + (size_t)(2 * c + 1) * kTile);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float4 x = ta[q], y = tb[q];
            ga[4 * q] += x.x; ga[4 * q + 1] += x.y; ga[4 * q + 2] += x.z; ga[4 * q + 3] += x.w;
            gb[4 * q] += y.x; gb[4 * q + 1] += y.y; gb[4 * q + 2] += y.z; gb[4 * q + 3] += y.w;
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += gb[r] * (ga[r] + L.bias);
    s = wave_sum(s * block_weight(threadIdx.x >> 6, bi == bj));
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        float t = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) t += red[w];
        L.out[n * L.pairs + p] = L.s2 * (bi == bj ? t : 2.0f * t);
    }
}

// sqnorm[n] of every layer with several pairs: one wave per (layer, sample)
// adds its pairs' values (lane l takes pairs l, l + 64, ..., then a butterfly)
__global__ __launch_bounds__(256) void ghost_pair_sum_kernel(const GhostGroup g)
{
    const GhostLayer &L = g.L[blockIdx.y];
    const i64 n = (i64)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (L.pairs == 1 || n >= g.N) return;
    const float *q = L.part + n * L.pairs;
    float s = 0.0f;
    for (int t = lane; t < L.pairs; t += kWave) s += q[t];
    s = wave_sum(s);
    if (lane == 0) L.sqnorm[n] = s;
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
struct Plan {
    int nb, pairs, chunks;
};

// chunks per unit for a launch of `units` (sample, pair) units: one when
// they fill the GPU, else enough to give every CU two workgroups, with at
// least 256 features per chunk on average
Plan layer_plan(i64 T, i64 din, i64 dout, i64 units)
{
    Plan pl;
    pl.nb = (int)ceil_div(T, kBT);
    pl.pairs = pl.nb * (pl.nb + 1) / 2;
    i64 c = units >= kFill ? 1 : ceil_div(kFill, units > 0 ? units : 1);
    const i64 cap = ceil_div(din + dout, 256);
    pl.chunks = (int)(c < cap ? c : cap);
    return pl;
}

i64 launch_units(const dp_ghost_layer *items, int count, i64 N)
{
    i64 u = 0;
    for (int i = 0; i < count; ++i)
        if (items[i].T > 0) {
            const i64 nb = ceil_div(items[i].T, kBT);
            u += N * (nb * (nb + 1) / 2);
        }
    return u;
}

size_t round256(size_t b) { return (b + 255) & ~(size_t)255; }

// workspace of one layer: the pair values (several pairs), then the chunks'
// partial tiles (several chunks)
size_t layer_ws(const Plan &pl, i64 N)
{
    size_t b = 0;
    if (pl.pairs > 1) b += round256((size_t)(N * pl.pairs) * sizeof(float));
    if (pl.chunks > 1) b += (size_t)(N * pl.pairs) * pl.chunks * 2 * kTile * sizeof(float);
    return b;
}

dp_status check_item(const dp_ghost_layer &it, i64 N)
{
    DPG_REQUIRE(it.T >= 0 && it.d_in >= 1 && it.d_out >= 1, DP_EINVAL);
    DPG_REQUIRE(it.T < (i64(1) << 20) && it.d_in < (i64(1) << 31) && it.d_out < (i64(1) << 31), DP_EINVAL);
    DPG_REQUIRE(N == 0 || it.sqnorm != nullptr, DP_EINVAL);
    DPG_REQUIRE(N * it.T == 0 || (it.A != nullptr && it.B != nullptr), DP_EINVAL);
    DPG_REQUIRE(it.T * (it.d_in > it.d_out ? it.d_in : it.d_out) < (i64(1) << 31), DP_EUNSUPPORTED);
    return DP_OK;
}

template <typename T, bool VEC>
void launch_gram(const GhostGroup &g, int blocks, hipStream_t stream)
{
    ghost_gram_kernel<T, VEC><<<(unsigned)blocks, kThreads, 0, stream>>>(g);
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_ghost_norm_linear_many_workspace_bytes(const dp_ghost_layer *items, int32_t count, int64_t N)
{
    if (items == nullptr || count <= 0 || N <= 0) return 0;
    const i64 units = launch_units(items, count, N);
    size_t b = 0;
    for (int i = 0; i < count; ++i) {
        const dp_ghost_layer &it = items[i];
        if (it.T <= 0 || it.d_in <= 0 || it.d_out <= 0) continue;
        b += layer_ws(layer_plan(it.T, it.d_in, it.d_out, units), N);
    }
    return b;
}

extern "C" dp_status dp_ghost_norm_linear_many(const dp_ghost_layer *items, int32_t count, dp_dtype dt, int64_t N,
                                               int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(count >= 0 && count <= 64 && (count == 0 || items != nullptr), DP_EINVAL);
    DPG_REQUIRE(N >= 0 && N < (i64(1) << 31), DP_EINVAL);
    for (int i = 0; i < count; ++i) {
        const dp_status st = check_item(items[i], N);
        if (st != DP_OK) return st;
    }
    const size_t need = dp_ghost_norm_linear_many_workspace_bytes(items, count, N);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0 || count == 0) return DP_OK;

    const i64 units = launch_units(items, count, N);
    const i64 pc = 16 / (i64)dtype_bytes(dt);
    const i64 F = kRowBytes / (i64)dtype_bytes(dt);
    GhostLayer lay[64];
    bool vec[64];
    int order[64], live = 0;
    char *w = (char *)ws;
    for (int i = 0; i < count; ++i) {
        const dp_ghost_layer &it = items[i];
        if (it.T == 0) {                         // an empty sum over positions: zero norms
            zero_fill(it.sqnorm, N, stream);
            continue;
        }
        const Plan pl = layer_plan(it.T, it.d_in, it.d_out, units);
        GhostLayer &L = lay[i];
        L.A = it.A;
        L.B = it.B;
        L.T = it.T;
        L.din = it.d_in;
        L.dout = it.d_out;
        L.nb = pl.nb;
        L.pairs = pl.pairs;
        L.chunks = pl.chunks;
        L.sa = (int)ceil_div(it.d_in, F);
        L.sb = (int)ceil_div(it.d_out, F);
        L.bias = it.bias ? 1.0f : 0.0f;
        L.s2 = it.scale * it.scale;
        L.sqnorm = it.sqnorm;
        L.part = nullptr;
        L.tiles = nullptr;
        if (pl.pairs > 1) {
            L.part = (float *)w;
            w += round256((size_t)(N * pl.pairs) * sizeof(float));
        }
        if (pl.chunks > 1) {
            L.tiles = (float *)w;
            w += (size_t)(N * pl.pairs) * pl.chunks * 2 * kTile * sizeof(float);
        }
        L.out = pl.pairs > 1 ? L.part : it.sqnorm;
        vec[i] = it.d_in % pc == 0 && it.d_out % pc == 0 && aligned(it.A, 16) && aligned(it.B, 16);
        order[live++] = i;
    }
    // more features per sample first (the longest units start first)
    for (int a = 1; a < live; ++a)
        for (int b = a; b > 0 && lay[order[b]].din + lay[order[b]].dout > lay[order[b - 1]].din +
                                                                           lay[order[b - 1]].dout; --b) {
            const int t = order[b];
            order[b] = order[b - 1];
            order[b - 1] = t;
        }

    // the Gram launches: the 16-byte class, then the element class, up to
    // kGroupMax layers per launch
    for (int cls = 0; cls < 2; ++cls) {
        const bool want_vec = cls == 0;
        GhostGroup g;
        g.N = N;
        g.count = 0;
        i64 blocks = 0;
        auto flush = [&]() -> dp_status {
            if (g.count == 0) return DP_OK;
            DPG_REQUIRE(blocks < (i64(1) << 31), DP_EUNSUPPORTED);
            if (dt == DP_BF16) {
                if (want_vec) launch_gram<uint16_t, true>(g, (int)blocks, stream);
                else launch_gram<uint16_t, false>(g, (int)blocks, stream);
            } else {
                if (want_vec) launch_gram<float, true>(g, (int)blocks, stream);
                else launch_gram<float, false>(g, (int)blocks, stream);
            }
            g.count = 0;
            blocks = 0;
            return DP_OK;
        };
        for (int a = 0; a < live; ++a) {
            const int i = order[a];
            if (vec[i] != want_vec) continue;
            GhostLayer &L = lay[i];
            L.blk0 = (int)blocks;
            blocks += 8 * (i64)(L.pairs * L.chunks) * ceil_div(N, 8);
            DPG_REQUIRE(blocks < (i64(1) << 31), DP_EUNSUPPORTED);
            g.L[g.count++] = L;
            if (g.count == kGroupMax) {
                const dp_status st = flush();
                if (st != DP_OK) return st;
            }
        }
        const dp_status st = flush();
        if (st != DP_OK) return st;
    }
    // several chunks: add them and form the pair values
    {
        GhostGroup g;
        g.N = N;
        g.count = 0;
        i64 blocks = 0;
        for (int a = 0; a <= live; ++a) {
            if (a < live) {
                GhostLayer &L = lay[order[a]];
                if (L.chunks == 1) continue;
                L.cblk0 = (int)blocks;
                blocks += N * L.pairs;
                g.L[g.count++] = L;
            }
            if (g.count > 0 && (g.count == kGroupMax || a == live)) {
                ghost_combine_kernel<<<(unsigned)blocks, kThreads, 0, stream>>>(g);
                g.count = 0;
                blocks = 0;
            }
        }
    }
    // several pairs: add them into sqnorm
    {
        GhostGroup g;
        g.N = N;
        g.count = 0;
        for (int a = 0; a <= live; ++a) {
            if (a < live) {
                const GhostLayer &L = lay[order[a]];
                if (L.pairs == 1) continue;
                g.L[g.count++] = L;
            }
            if (g.count > 0 && (g.count == kGroupMax || a == live)) {
                const dim3 grid((unsigned)ceil_div(N, 4), (unsigned)g.count);
                ghost_pair_sum_kernel<<<grid, 256, 0, stream>>>(g);
                g.count = 0;
            }
        }
    }
    return launch_status();
}

extern "C" size_t dp_ghost_norm_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in, int64_t d_out)
{
    if (N <= 0 || T <= 0 || d_in <= 0 || d_out <= 0) return 0;
    dp_ghost_layer it{};
    it.T = T;
    it.d_in = d_in;
    it.d_out = d_out;
    return dp_ghost_norm_linear_many_workspace_bytes(&it, 1, N);
}

extern "C" dp_status dp_ghost_norm_linear(const void *A, const void *B, dp_dtype dt, int64_t N, int64_t T,
                                          int64_t d_in, int64_t d_out, float scale, int32_t bias, float *sqnorm,
                                          int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && N < (i64(1) << 31), DP_EINVAL);
    dp_ghost_layer it;
    it.A = A;
    it.B = B;
    it.T = T;
    it.d_in = d_in;
    it.d_out = d_out;
    it.scale = scale;
    it.bias = bias;
    it.sqnorm = sqnorm;
    return dp_ghost_norm_linear_many(&it, 1, dt, N, status, ws, ws_bytes, stream);
}
