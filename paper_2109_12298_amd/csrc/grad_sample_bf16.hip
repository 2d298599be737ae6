// Per-sample gradients of a Linear layer over a sequence with bf16 inputs
// (appendix "Vectorized Computation": the per-sample gradient is B_n^T A_n,
// summed over the extra dimension):
//   gW_n[i][j] = s * sum_t B_n[t][i] * A_n[t][j],   gb_n[i] = s * sum_t B_n[t][i]
// in fp32, on v_mfma_f32_32x32x16_bf16, with each (sample, tile)'s squared
// norm written as partials (one per wave) from the values it stores.
//
// The layer's per-sample gradients are N * d_out * d_in fp32 values, written
// once: the kernel is bound by that write, not by the MFMAs (a 256 x 128
// tile is 4M multiply-adds per 128 KB stored).  So a workgroup owns one
// 256 (j) x 128 (i) tile for a run of consecutive samples, and its operand
// loads never stop: the rows of consecutive samples are consecutive rows of
// A [N*T][d_in] and B [N*T][d_out], so the 32-row stages (bf16_stage.hpp:
// direct-to-LDS loads, three stages deep, transposing operand reads) run
// straight through the sample boundaries.  At the end of each sample the
// accumulators are scaled and stored and the next sample's MFMAs start on
// operands already in LDS, so the stores of one sample drain while the next
// is multiplied.  Needs T % 32 == 0 and d_in, d_out multiples of 8.
//
// Balance.  Every (sample, tile) unit costs the same, and two workgroups fit
// a CU, so 512 run at once.  The run length p is chosen so that the units
// divide into whole rounds of 512 workgroups: a launch of 1152 two-sample
// runs would leave three quarters of the machine idle for its third round.
// The grouped launch (bf16_grad_group_kernel) takes every such layer of a
// step at once, its workgroups the concatenation of the layers' runs, so the
// layers' last rounds fill each other's idle slots.
#include "bf16_stage.hpp"
#include "grad_sample_bf16.hpp"

namespace dpg {
namespace {

using namespace bf16s;

// Tile configuration: four waves in a 2 x 2 layout, each owning FM x FN
// blocks of 32 x 32, so the workgroup tile is 64*FM (j) x 64*FN (i).
template <int FM_, int FN_, int STAGES_>
struct GsCfg {
    static constexpr int FM = FM_, FN = FN_, STAGES = STAGES_;
    static constexpr int BMJ = 64 * FM, BNI = 64 * FN;
    static constexpr int WAVES = 4, THREADS = 256;
    typedef StagePlan<BMJ, BNI, WAVES> Plan;
    static constexpr int BIAS_ROWS = BK * 32 / THREADS;    // stage rows per thread in the bias sums
    static constexpr int STORES = FM * FN * 4;              // float4 stores per wave per sample
};
// the configuration the entry point uses
typedef GsCfg<4, 2, 3> Gs;

// The run of one workgroup: tile `tile` of a layer (tiles_m tiles along j)
// for samples s0 .. s0+ns-1; partial[n][tile][wave] receives each sample's
// squared-norm partials (if partial is not NULL).
template <typename Cfg>
__device__ __forceinline__ void grad_sample_run(const uint16_t *__restrict__ A, const uint16_t *__restrict__ B,
                                                i64 T, i64 din, i64 dout, int tiles_m, int tiles, int tile, i64 s0,
                                                int ns, float scale, float *__restrict__ gW,
                                                float *__restrict__ gb, float *__restrict__ partial)
{
    typedef typename Cfg::Plan Plan;
    constexpr int FM = Cfg::FM, FN = Cfg::FN, BMJ = Cfg::BMJ, BNI = Cfg::BNI, kStages = Cfg::STAGES;
    constexpr int kThreads = Cfg::THREADS, kWaves = Cfg::WAVES;
    constexpr int A_ROW = Plan::A_ROW, B_ROW = Plan::B_ROW, A_BYTES = Plan::A_BYTES;
    constexpr int STAGE_BYTES = Plan::STAGE_BYTES, BIAS_ROWS = Cfg::BIAS_ROWS;
    typedef Frag<FM, FN> WaveFrag;
    auto load_wave_frag = [&](const char *L, int ks, int wj, int wi, int lane, WaveFrag &f) {
        load_frag<FM, FN, A_ROW, B_ROW, A_BYTES>(L, ks, wj, wi, lane, f);
    };
    __shared__ __attribute__((aligned(1024))) char smem[kStages * STAGE_BYTES];
    __shared__ float bred[kThreads / 32][BNI];
    const int tn = tile / tiles_m, tm = tile % tiles_m;
    const i64 m0 = (i64)tm * BMJ, n0 = (i64)tn * BNI;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wj = (wave >> 1) * 32 * FM, wi = (wave & 1) * 32 * FN;
    const bool do_bias = gb != nullptr && tm == 0;
    const bool full_tile = m0 + BMJ <= din && n0 + BNI <= dout;
    const int sps = (int)(T / BK);                 // stages per sample
    const int nst = ns * sps;
    const uint16_t *Ab = A + s0 * T * din;         // this block's first sample
    const uint16_t *Bb = B + s0 * T * dout;
    const uint32_t lds0 = lds_addr(smem);
    const Plan sp(din, dout, m0, n0, wave, lane);

    f32x16_t acc[FM][FN];
#pragma unroll
    for (int x = 0; x < FM; ++x)
#pragma unroll
        for (int y = 0; y < FN; ++y)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.0f;
    // bias: thread sums 4 consecutive columns (group cg) over rows
    // BIAS_ROWS*rg .. of every stage of the sample
    const int cg = tid & 31, rg = tid >> 5;
    float bsum[4] = {0.0f, 0.0f, 0.0f, 0.0f};

#pragma unroll
    for (int c = 0; c < kStages - 1; ++c)
        if (c < nst) sp.issue(Ab, Bb, din, dout, (i64)c * BK, lds0 + c * STAGE_BYTES);
    wait_vmcnt_rt((nst - 1 < kStages - 2 ? nst - 1 : kStages - 2) * Plan::LOADS);   // stage 0 has landed
    stage_barrier();
    if (kStages - 1 < nst) sp.issue(Ab, Bb, din, dout, (i64)(kStages - 1) * BK, lds0 + (kStages - 1) * STAGE_BYTES);

    // the end of sample n: store s * acc (and the bias), the wave's squared-norm
    // partial, and clear the accumulators
    auto finish_sample = [&](i64 n) {
        float sq = 0.0f;
        float *G = gW + n * dout * din;
        const int li = lane & 31, kg = lane >> 5;
#pragma unroll
        for (int x = 0; x < FM; ++x)
#pragma unroll
            for (int y = 0; y < FN; ++y) {
                const i64 i = n0 + wi + 32 * y + li;
#pragma unroll
                for (int rb = 0; rb < 4; ++rb) {
                    const i64 j = m0 + wj + 32 * x + 8 * rb + 4 * kg;
                    const float g0 = scale * acc[x][y][4 * rb + 0], g1 = scale * acc[x][y][4 * rb + 1];
                    const float g2 = scale * acc[x][y][4 * rb + 2], g3 = scale * acc[x][y][4 * rb + 3];
                    if (i < dout && j < din) {   // d_in % 8 == 0: the four j are all in or all out
                        *reinterpret_cast<float4 *>(G + i * din + j) = make_float4(g0, g1, g2, g3);
                        sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
                    }
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.0f;
            }
        if (do_bias) {
            // the row groups' column sums, added in row-group order
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                bred[rg][4 * cg + q] = bsum[q];
                bsum[q] = 0.0f;
            }
            __syncthreads();
            if (tid < BNI && n0 + tid < dout) {
                float b = 0.0f;
#pragma unroll
                for (int r = 0; r < kThreads / 32; ++r) b += bred[r][tid];
                b *= scale;
                gb[n * dout + n0 + tid] = b;
                sq += b * b;
            }
            __syncthreads();
        }
        sq = wave_sum(sq);
        if (partial && lane == 0) partial[n * (i64)tiles * kWaves + (i64)tile * kWaves + wave] = sq;
    };

    // fa: k-step 0 of the current stage, fb: k-step 1 (read during the MFMAs
    // of the previous k-step); the last stage is peeled so that every loop
    // trip has the same straight read/MFMA blocks
    WaveFrag fa, fb;
    int ends = 0;            // bit k: the iteration k+1 back ended a sample (and stored it)
    int in_sample = 0;
    i64 n = s0;
    if (nst > 0) load_wave_frag(smem, 0, wj, wi, lane, fa);
    for (int c = 0; c + 1 < nst; ++c) {
        const char *L = smem + (c % kStages) * STAGE_BYTES;
        if (do_bias) {
#pragma unroll
            for (int r = 0; r < BIAS_ROWS; ++r) {
                const uint2 v = *reinterpret_cast<const uint2 *>(L + A_BYTES + swz(BIAS_ROWS * rg + r, 4 * cg, B_ROW));
                bsum[0] += __uint_as_float(v.x << 16);
                bsum[1] += __uint_as_float(v.x & 0xffff0000u);
                bsum[2] += __uint_as_float(v.y << 16);
                bsum[3] += __uint_as_float(v.y & 0xffff0000u);
            }
        }
        load_wave_frag(L, 1, wj, wi, lane, fb);
        mma(fa, acc);
        interleave_reads_with_mfma<FM, FN>();
        // stage c+1 has landed once at most the vector-memory operations issued
        // after its loads remain: the loads of up to two later stages and, in
        // a full tile, the 16 stores per wave of each sample that ended in the
        // last three iterations (a partial tile counts none of its stores and
        // so waits for them too)
        {
            const int later = nst - 2 - c < kStages - 2 ? nst - 2 - c : kStages - 2;
            const int stores = full_tile ? Cfg::STORES * __builtin_popcount(ends & ((1 << (kStages - 1)) - 1)) : 0;
            const int n_after = later * Plan::LOADS + stores;
            wait_vmcnt_rt(n_after < 63 ? n_after : 63);   // capping only waits longer
        }
        wait_lgkmcnt0();                               // this wave's reads of stage c are done
        stage_barrier();
        if (c + kStages < nst)
            sp.issue(Ab, Bb, din, dout, (i64)(c + kStages) * BK, lds0 + (uint32_t)(c % kStages) * STAGE_BYTES);
        load_wave_frag(smem + ((c + 1) % kStages) * STAGE_BYTES, 0, wj, wi, lane, fa);
        mma(fb, acc);
        interleave_reads_with_mfma<FM, FN>();
        ends <<= 1;
        if (++in_sample == sps) {
            finish_sample(n);
            in_sample = 0;
            ++n;
            ends |= 1;
        }
    }
    if (nst > 0) {
        const char *L = smem + ((nst - 1) % kStages) * STAGE_BYTES;
        if (do_bias) {
#pragma unroll
            for (int r = 0; r < BIAS_ROWS; ++r) {
                const uint2 v = *reinterpret_cast<const uint2 *>(L + A_BYTES + swz(BIAS_ROWS * rg + r, 4 * cg, B_ROW));
                bsum[0] += __uint_as_float(v.x << 16);
                bsum[1] += __uint_as_float(v.x & 0xffff0000u);
                bsum[2] += __uint_as_float(v.y << 16);
                bsum[3] += __uint_as_float(v.y & 0xffff0000u);
            }
        }
        load_wave_frag(L, 1, wj, wi, lane, fb);
        mma(fa, acc);
        mma(fb, acc);
        finish_sample(n);
    }
}

// Single layer: block b = (run of samples, tile); consecutive blocks share
// the run and walk the tiles (neighbouring tiles share operand rows in one
// XCD's L2).
template <typename Cfg>
__global__ __launch_bounds__(Cfg::THREADS, 2) void bf16_grad_sample_kernel(
    const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, i64 N, i64 T, i64 din, i64 dout, int tiles_m,
    int tiles, int per_block, float scale, float *__restrict__ gW, float *__restrict__ gb,
    float *__restrict__ partial)
{
    const i64 blk = xcd_swizzle(blockIdx.x, gridDim.x);
    const int tile = (int)(blk % tiles);
    const i64 s0 = (blk / tiles) * per_block;
    const int ns = (int)(s0 + per_block < N ? per_block : N - s0);   // samples of this block
    grad_sample_run<Cfg>(A, B, T, din, dout, tiles_m, tiles, tile, s0, ns, scale, gW, gb, partial);
}

struct GsItem {
    const uint16_t *A, *B;
    float *gW, *gb, *partial, *sqnorm;
    i64 din, dout, T;
    float scale;
    int tiles_m, tiles;
};

struct GsGroup {
    int count;
    int per;                          // samples per run
    i64 N;
    int blk0[kBf16GroupMax + 1];      // first block of each layer
    GsItem it[kBf16GroupMax];
};

// Several layers: the blocks are the concatenation of every layer's (run,
// tile) blocks; a block finds its layer in the prefix table.
template <typename Cfg>
__global__ __launch_bounds__(Cfg::THREADS, 2) void bf16_grad_group_kernel(const GsGroup g)
{
    const int blk = (int)xcd_swizzle(blockIdx.x, gridDim.x);
    int k = 0;
    while (k + 1 < g.count && g.blk0[k + 1] <= blk) ++k;
    const GsItem &it = g.it[k];
    const int local = blk - g.blk0[k];
    const int tile = local % it.tiles;
    const i64 s0 = (i64)(local / it.tiles) * g.per;
    const int ns = (int)(s0 + g.per < g.N ? g.per : g.N - s0);
    grad_sample_run<Cfg>(it.A, it.B, it.T, it.din, it.dout, it.tiles_m, it.tiles, tile, s0, ns, it.scale, it.gW,
                         it.gb, it.partial);
}

// One wave per (layer, sample): sqnorm[n] = the sample's partials added in
// tile and wave order (lane l takes partials l, l+64, ..., then a fixed
// butterfly), as sum_partials does for one layer.
__global__ __launch_bounds__(256) void bf16_group_sqnorm_kernel(const GsGroup g)
{
    const GsItem &it = g.it[blockIdx.y];
    const i64 n = (i64)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (it.sqnorm == nullptr || n >= g.N) return;
    const int parts = it.tiles * Gs::WAVES;
    const float *p = it.partial + n * parts;
    float s = 0.0f;
    for (int t = lane; t < parts; t += kWave) s += p[t];
    s = wave_sum(s);
    if (lane == 0) it.sqnorm[n] = s;
}

constexpr int kSlots = 2 * 256;      // resident workgroups: two per CU, 256 CUs

// Samples per run for `tiles` tiles (all layers) of N samples: the fewest
// rounds of kSlots workgroups times the run length, ties to the longer run
// (fewer pipeline starts).
int run_length(i64 N, i64 tiles)
{
    int best = 1;
    i64 best_cost = -1;
    for (int p = 1; p <= 8; ++p) {
        const i64 cost = ceil_div(tiles * ceil_div(N, p), kSlots) * p;
        if (best_cost < 0 || cost <= best_cost) {
            best_cost = cost;
            best = p;
        }
    }
    return best;
}

}  // namespace

bool bf16_staged_ok(const void *A, const void *B, const void *gW, i64 N, i64 T, i64 din, i64 dout)
{
    return T >= BK && T % BK == 0 && din % 8 == 0 && dout % 8 == 0 && aligned(A, 16) && aligned(B, 16) &&
           aligned(gW, 16) && T * (din > dout ? din : dout) < (i64(1) << 31) && N < (i64(1) << 40) &&
           N * ceil_div(din, Gs::BMJ) * ceil_div(dout, Gs::BNI) < (i64(1) << 30);
}

int bf16_staged_parts(i64 din, i64 dout)
{
    return (int)(ceil_div(din, Gs::BMJ) * ceil_div(dout, Gs::BNI)) * Gs::WAVES;
}

void bf16_grad_sample_staged(const void *A, const void *B, i64 N, i64 T, i64 din, i64 dout, float scale, float *gW,
                             float *gb, float *partial, hipStream_t stream)
{
    const int tiles_m = (int)ceil_div(din, Gs::BMJ);
    const int tiles = tiles_m * (int)ceil_div(dout, Gs::BNI);
    const int per = run_length(N, tiles);
    const i64 runs = ceil_div(N, per);
    bf16_grad_sample_kernel<Gs><<<(unsigned)(runs * tiles), Gs::THREADS, 0, stream>>>(
        (const uint16_t *)A, (const uint16_t *)B, N, T, din, dout, tiles_m, tiles, per, scale, gW, gb, partial);
}

void bf16_grad_sample_group(const Bf16GroupLayer *layers, int count, i64 N, hipStream_t stream)
{
    if (count <= 0 || N <= 0) return;
    GsGroup g;
    g.count = count;
    g.N = N;
    i64 tiles = 0;
    bool norms = false;
    for (int k = 0; k < count; ++k) {
        const Bf16GroupLayer &L = layers[k];
        GsItem &it = g.it[k];
        it.A = (const uint16_t *)L.A;
        it.B = (const uint16_t *)L.B;
        it.gW = L.gW;
        it.gb = L.gb;
        it.sqnorm = L.sqnorm;
        it.partial = L.sqnorm ? L.partial : nullptr;
        it.din = L.din;
        it.dout = L.dout;
        it.T = L.T;
        it.scale = L.scale;
        it.tiles_m = (int)ceil_div(L.din, Gs::BMJ);
        it.tiles = it.tiles_m * (int)ceil_div(L.dout, Gs::BNI);
        tiles += it.tiles;
        norms = norms || L.sqnorm != nullptr;
    }
    g.per = run_length(N, tiles);
    const i64 runs = ceil_div(N, g.per);
    int blocks = 0;
    for (int k = 0; k < count; ++k) {
        g.blk0[k] = blocks;
        blocks += (int)(runs * g.it[k].tiles);
    }
    for (int k = count; k <= kBf16GroupMax; ++k) g.blk0[k] = blocks;
    for (int k = count; k < kBf16GroupMax; ++k) g.it[k] = g.it[0];
    bf16_grad_group_kernel<Gs><<<(unsigned)blocks, Gs::THREADS, 0, stream>>>(g);
    if (norms) bf16_group_sqnorm_kernel<<<dim3((unsigned)ceil_div(N, 4), (unsigned)count), 256, 0, stream>>>(g);
}

}  // namespace dpg
