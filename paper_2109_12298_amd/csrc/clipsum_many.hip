// Grouped fused clipped sum of bf16 Linear layers over a sequence, on
// v_mfma_f32_32x32x16_bf16.
//
// For every layer of the group (section 1's clip-then-sum; appendix
// "Vectorized Computation" for the per-sample product):
//   S_W[i][j] = s * sum_n c_n * sum_t B_n[t][i] * A_n[t][j]
//   S_b[i]    = s * sum_n c_n * sum_t B_n[t][i]
// with c_n = min(1, C / (norm_n + 1e-6)).  This is a GEMM S_W = B^T diag(c) A
// whose K runs over all N*T (sample, position) rows of A [N*T][d_in] and
// B [N*T][d_out]; no per-sample gradient is read.
//
// One launch covers every layer: workgroup b finds its layer in a prefix
// table of tile counts, so small layers (768 x 768) and large ones
// (3072 x 768) share the machine.  Each workgroup (four waves, one per SIMD)
// owns a 256 (j) x 128 (i) output tile and the whole K range of up to 4000
// samples, so no partial sums leave the chip; larger batches run as several
// launches, each adding its samples to the sums the previous one stored.
//
// Clip factors with a single set of accumulators.  While sample n is added
// the accumulators hold S / c_n.  When sample n+1 begins they are multiplied
// by c_n / c_{n+1} (one VALU multiply per accumulator per sample, issued
// before the new sample's first MFMAs), and the final tile is multiplied by
// s * c_last.  Every operand stays in bf16 exactly as stored; c
// is applied in fp32.  The accumulators never overflow for finite norms:
// |S| <= n * C because every clipped gradient has norm <= C, so
// |S / c_n| <= n * (norm_n + 1e-6).  A sample whose factor underflows to 0
// contributes nothing and is skipped; a NaN factor (non-finite norm) turns
// the whole sum to NaN, as the column reduction does.  The clip factors of
// the launch's samples (and their reciprocals) are computed once per
// workgroup into LDS.
//
// Operand staging.  Both operands are K-major in memory ([row][feature]).
// Each 32-row stage of both tiles is copied straight from global memory into
// LDS by global_load_lds_dwordx4 (16 bytes per lane, 1 KB per wave
// instruction, no VGPR round trip), four stages deep, so up to three stages
// of loads are in flight while one is multiplied.  Inside a row, 16-byte chunk q
// is stored at chunk position q ^ (4 * (row & 3)); the transposing LDS read
// ds_read_b64_tr_b16 that forms each MFMA operand (eight consecutive rows of
// one feature per lane) then touches four rows whose 64-byte pieces fall in
// four different quarters of the 256-byte bank window: no bank conflicts.
// Each k-step's twelve operand reads (for the next k-step) are issued between
// its eight MFMAs.
#include "bf16_stage.hpp"
#include "clipsum_many.hpp"

#include <type_traits>

namespace dpg {
namespace {

using namespace bf16s;

constexpr int BMJ = 256;                         // j (d_in) per tile
constexpr int BNI = 128;                         // i (d_out) per tile
constexpr int kStages = 4;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
typedef StagePlan<BMJ, BNI, kWaves> Plan;
constexpr int A_ROW = Plan::A_ROW, B_ROW = Plan::B_ROW;
constexpr int A_BYTES = Plan::A_BYTES;           // 16 KB
constexpr int STAGE_BYTES = Plan::STAGE_BYTES;   // 24 KB
constexpr int BIAS_ROWS = BK * 32 / kThreads;     // stage rows per thread in the bias sums
constexpr int kChunkN = 4000;                    // samples per launch (clip factors in LDS)
static_assert(kStages * STAGE_BYTES + 2 * kChunkN * 4 + 256 <= 160 * 1024, "LDS budget");
typedef Frag<4, 2> WaveFrag;                     // a wave's 128 (j) x 64 (i) part of the tile

struct Item {
    const uint16_t *A;
    const uint16_t *B;
    float *W;
    float *b;
    i64 din, dout, T;
    float scale;
    int tiles_m;
};

struct Group {
    int count;
    int N;                 // samples of this launch (<= kChunkN)
    int accumulate;        // add to the sums already stored (later launches of a large batch)
    int blk0[kClipManyMax + 1];
    Item it[kClipManyMax];
};

__device__ __forceinline__ int find_item(const int *blk0, int count, int b)
{
    int p = 0;
    while (p + 1 < count && blk0[p + 1] <= b) ++p;
    return p;
}

__device__ __forceinline__ void load_wave_frag(const char *L, int ks, int wj, int wi, int lane, WaveFrag &f)
{
    load_frag<4, 2, A_ROW, B_ROW, A_BYTES>(L, ks, wj, wi, lane, f);
}

// Pipeline.  Stage c (32 rows of A and B) lives in LDS buffer c % 4.  A wave
// multiplies a stage as two k-steps; the operands of each k-step are read
// from LDS during the previous k-step's MFMAs (two register sets, used in
// turn).  Between the two k-steps of stage c the waves meet at a barrier once
// stage c+1 has landed; stage c's buffer is then free and takes the loads of
// stage c+4, and the second k-step's MFMAs overlap the reads of stage c+1's
// first k-step.
__global__ __launch_bounds__(kThreads, 1) void bf16_clipsum_many_kernel(Group g, const float *__restrict__ norm,
                                                                        float C)
{
    __shared__ __attribute__((aligned(1024))) char smem[kStages * STAGE_BYTES];
    __shared__ float cf[kChunkN], icf[kChunkN];      // clip factors of the launch's samples, and 1/c
    const int b = (int)xcd_swizzle(blockIdx.x, gridDim.x);
    const int p = find_item(g.blk0, g.count, b);
    const Item it = g.it[p];
    const int tile = b - g.blk0[p];
    const int tn = tile / it.tiles_m, tm = tile % it.tiles_m;   // neighbouring blocks share the i-tile
    const i64 m0 = (i64)tm * BMJ, n0 = (i64)tn * BNI;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wj = (wave >> 1) * 128, wi = (wave & 1) * 64;
    const bool do_bias = it.b != nullptr && tm == 0;
    const int sps = (int)(it.T / BK);              // stages per sample
    const int nst = g.N * sps;                     // stages
    // LDS byte address of the stage buffers (what M0 takes)
    const uint32_t lds0 = lds_addr(smem);
    const Plan sp(it.din, it.dout, m0, n0, wave, lane);

    int zero = 0;
    for (int n = tid; n < g.N; n += kThreads) {
        const float c = clip_factor(norm[n], C);
        cf[n] = c;
        icf[n] = 1.0f / c;
        zero |= c == 0.0f;
    }
    // a factor that underflowed to 0 needs the slower loop that skips samples
    const bool any_zero = __syncthreads_or(zero) != 0;

    f32x16_t acc[4][2];
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.0f;
    // bias: thread sums 4 consecutive columns (group cg) over BIAS_ROWS rows
    // of each stage (row group rg), per sample (bcur), then weighted into btot
    const int cg = tid & 31, rg = tid >> 5;
    float bcur[4] = {0.0f, 0.0f, 0.0f, 0.0f}, btot[4] = {0.0f, 0.0f, 0.0f, 0.0f};

#pragma unroll
    for (int c = 0; c < kStages - 1; ++c)
        if (c < nst) sp.issue(it.A, it.B, it.din, it.dout, (i64)c * BK, lds0 + c * STAGE_BYTES);
    wait_stages_after<Plan::LOADS>(nst - 1);   // stage 0 has landed
    stage_barrier();
    if (kStages - 1 < nst)
        sp.issue(it.A, it.B, it.din, it.dout, (i64)(kStages - 1) * BK, lds0 + (kStages - 1) * STAGE_BYTES);

    float c_cur = 1.0f;      // the accumulators hold S / c_cur
    float c_bias = 0.0f;     // clip factor of the sample whose bias rows are in bcur
    bool skip = false;       // the current sample's factor is 0: it adds nothing
    int in_sample = 0;       // stage index within the current sample
    int n = 0;               // sample of the stage being multiplied

    // per-stage work before the MFMAs: a new sample's rescale, and the bias rows
    auto begin_stage = [&](const char *L, auto zero_tag) {
        constexpr bool kZero = decltype(zero_tag)::value;
        if (in_sample == 0) {
            // a new sample: rescale the accumulators from S / c_prev to S / c_n
            const float cn = cf[n];
            skip = kZero && cn == 0.0f;
            if (!skip) {
                const float ratio = c_cur * icf[n];
#pragma unroll
                for (int x = 0; x < 4; ++x)
#pragma unroll
                    for (int y = 0; y < 2; ++y)
#pragma unroll
                        for (int r = 0; r < 16; ++r) acc[x][y][r] *= ratio;
                c_cur = cn;
            }
            if (do_bias) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    btot[q] += c_bias * bcur[q];
                    bcur[q] = 0.0f;
                }
                c_bias = cn;
            }
        }
        if (do_bias) {
#pragma unroll
            for (int r = 0; r < BIAS_ROWS; ++r) {
                const int t = BIAS_ROWS * rg + r;
                const uint2 v = *reinterpret_cast<const uint2 *>(L + A_BYTES + swz(t, 4 * cg, B_ROW));
                bcur[0] += __uint_as_float(v.x << 16);
                bcur[1] += __uint_as_float(v.x & 0xffff0000u);
                bcur[2] += __uint_as_float(v.y << 16);
                bcur[3] += __uint_as_float(v.y & 0xffff0000u);
            }
        }
    };
    auto next_stage = [&](int c) {
        wait_stages_after<Plan::LOADS>(nst - 2 - c);   // stage c+1 has landed
        wait_lgkmcnt0();                  // this wave's reads of stage c are done
        stage_barrier();
        if (c + kStages < nst)
            sp.issue(it.A, it.B, it.din, it.dout, (i64)(c + kStages) * BK,
                     lds0 + (uint32_t)(c % kStages) * STAGE_BYTES);
    };
    auto end_stage = [&]() {
        if (++in_sample == sps) {
            in_sample = 0;
            ++n;
        }
    };

    // the main loop; kZero: some factor is 0 and its samples are skipped (a
    // branch around the MFMAs, which the common loop does without, so that
    // each k-step is one straight block whose reads and MFMAs the scheduler
    // can interleave).  fa: k-step 0 of the current stage, fb: k-step 1.  The
    // last stage is peeled so that every loop trip has the same blocks.
    auto run = [&](auto zero_tag) {
        constexpr bool kZero = decltype(zero_tag)::value;
        WaveFrag fa, fb;
        if (nst > 0) load_wave_frag(smem, 0, wj, wi, lane, fa);
        for (int c = 0; c + 1 < nst; ++c) {
            const char *L = smem + (c % kStages) * STAGE_BYTES;
            begin_stage(L, zero_tag);
            load_wave_frag(L, 1, wj, wi, lane, fb);
            if (!kZero || !skip) mma(fa, acc);
            interleave_reads_with_mfma<4, 2>();
            next_stage(c);
            load_wave_frag(smem + ((c + 1) % kStages) * STAGE_BYTES, 0, wj, wi, lane, fa);
            if (!kZero || !skip) mma(fb, acc);
            interleave_reads_with_mfma<4, 2>();
            end_stage();
        }
        if (nst > 0) {
            const char *L = smem + ((nst - 1) % kStages) * STAGE_BYTES;
            begin_stage(L, zero_tag);
            load_wave_frag(L, 1, wj, wi, lane, fb);
            if (!kZero || !skip) {
                mma(fa, acc);
                mma(fb, acc);
            }
            end_stage();
        }
    };
    if (any_zero)
        run(std::true_type{});
    else
        run(std::false_type{});
    if (do_bias) {
#pragma unroll
        for (int q = 0; q < 4; ++q) btot[q] += c_bias * bcur[q];
    }

    // store S (or add it to the stored sums of the earlier samples)
    const float fs = it.scale * c_cur;
    const int li = lane & 31, kg = lane >> 5;
#pragma unroll
    for (int x = 0; x < 4; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const i64 i = n0 + wi + 32 * y + li;
            if (i >= it.dout) continue;
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const i64 j = m0 + wj + 32 * x + 8 * rb + 4 * kg;
                if (j >= it.din) continue;   // d_in % 8 == 0: the four j are all in or all out
                float4 v = make_float4(fs * acc[x][y][4 * rb + 0], fs * acc[x][y][4 * rb + 1],
                                       fs * acc[x][y][4 * rb + 2], fs * acc[x][y][4 * rb + 3]);
                float4 *dst = reinterpret_cast<float4 *>(it.W + i * it.din + j);
                if (g.accumulate) {
                    const float4 o = *dst;
                    v = make_float4(o.x + v.x, o.y + v.y, o.z + v.z, o.w + v.w);
                }
                *dst = v;
            }
        }
    if (do_bias) {
        // the row groups' column sums, added in row-group order
        float *red = reinterpret_cast<float *>(smem);
        __syncthreads();
#pragma unroll
        for (int q = 0; q < 4; ++q) red[rg * BNI + 4 * cg + q] = btot[q];
        __syncthreads();
        if (tid < BNI && n0 + tid < it.dout) {
            float s = 0.0f;
#pragma unroll
            for (int r = 0; r < kThreads / 32; ++r) s += red[r * BNI + tid];
            s *= it.scale;
            float *dst = it.b + n0 + tid;
            *dst = g.accumulate ? *dst + s : s;
        }
    }
}

}  // namespace

bool clip_many_item_ok(const void *A, const void *B, const float *W, const float *bsum, i64 N, i64 T, i64 din,
                       i64 dout)
{
    (void)N;
    return T >= BK && T % BK == 0 && (T / BK) * kChunkN < (i64(1) << 31) && din % 8 == 0 && dout % 8 == 0 &&
           aligned(A, 16) && aligned(B, 16) && aligned(W, 16) && (bsum == nullptr || aligned(bsum, 4));
}

void clip_many_launch(const ClipManyItem *items, int count, i64 N, const float *norm, float C, hipStream_t stream)
{
    // samples in chunks of kChunkN, each launch adding to the sums of the previous ones
    for (i64 s0 = 0; s0 < N; s0 += kChunkN) {
        Group g;
        g.count = count;
        g.N = (int)(N - s0 < kChunkN ? N - s0 : kChunkN);
        g.accumulate = s0 > 0;
        int blocks = 0;
        for (int k = 0; k < count; ++k) {
            const ClipManyItem &s = items[k];
            Item &d = g.it[k];
            d.A = (const uint16_t *)s.A + s0 * s.T * s.din;
            d.B = (const uint16_t *)s.B + s0 * s.T * s.dout;
            d.W = s.W;
            d.b = s.b;
            d.din = s.din;
            d.dout = s.dout;
            d.T = s.T;
            d.scale = s.scale;
            d.tiles_m = (int)ceil_div(s.din, BMJ);
            g.blk0[k] = blocks;
            blocks += d.tiles_m * (int)ceil_div(s.dout, BNI);
        }
        g.blk0[count] = blocks;
        if (blocks == 0) return;
        bf16_clipsum_many_kernel<<<(unsigned)blocks, kThreads, 0, stream>>>(g, norm + s0, C);
    }
}

}  // namespace dpg

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
using namespace dpg;

namespace {

bool grouped(const dp_linear_clip &x, dp_dtype dt, int64_t N)
{
    return dt == DP_BF16 && N > 0 && clip_many_item_ok(x.A, x.B, x.sumW, x.sumb, N, x.T, x.d_in, x.d_out);
}

}  // namespace

extern "C" size_t dp_clip_accumulate_linear_many_workspace_bytes(const dp_linear_clip *items, int32_t count,
                                                                 dp_dtype dt, int64_t N)
{
    size_t need = 0;
    if (items == nullptr || count <= 0) return 0;
    for (int32_t k = 0; k < count; ++k) {
        const dp_linear_clip &x = items[k];
        if (grouped(x, dt, N)) continue;
        const size_t w = dp_clip_accumulate_linear_workspace_bytes(N, x.T, x.d_in, x.d_out, dt);
        if (w > need) need = w;
    }
    return need;
}

extern "C" dp_status dp_clip_accumulate_linear_many(const dp_linear_clip *items, int32_t count, dp_dtype dt,
                                                    int64_t N, const float *norm, float C, int32_t *status,
                                                    void *ws, size_t ws_bytes, hipStream_t stream)
{
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(count >= 0 && (count == 0 || items != nullptr), DP_EINVAL);
    DPG_REQUIRE(N >= 0 && N < (i64(1) << 40), DP_EINVAL);
    DPG_REQUIRE(N == 0 || norm != nullptr, DP_EINVAL);
    DPG_REQUIRE(C > 0.0f, DP_EINVAL);
    for (int32_t k = 0; k < count; ++k) {
        const dp_linear_clip &x = items[k];
        DPG_REQUIRE(x.T >= 0 && x.d_in >= 1 && x.d_out >= 1 && x.T < (i64(1) << 40), DP_EINVAL);
        DPG_REQUIRE(N * x.T == 0 || (x.A != nullptr && x.B != nullptr), DP_EINVAL);
        DPG_REQUIRE(x.sumW != nullptr, DP_EINVAL);
    }
    const size_t need = dp_clip_accumulate_linear_many_workspace_bytes(items, count, dt, N);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);

    ClipManyItem batch[kClipManyMax];
    int nb = 0;
    for (int32_t k = 0; k < count; ++k) {
        const dp_linear_clip &x = items[k];
        if (!grouped(x, dt, N)) {
            const dp_status st = dp_clip_accumulate_linear(x.A, x.B, dt, N, x.T, x.d_in, x.d_out, x.scale, norm, C,
                                                           x.sumW, x.sumb, status, ws, ws_bytes, stream);
            if (st != DP_OK) return st;
            continue;
        }
        batch[nb++] = ClipManyItem{x.A, x.B, x.sumW, x.sumb, x.d_in, x.d_out, x.T, x.scale};
        if (nb == kClipManyMax) {
            clip_many_launch(batch, nb, N, norm, C, stream);
            nb = 0;
        }
    }
    if (nb > 0) clip_many_launch(batch, nb, N, norm, C, stream);
    return launch_status();
}
