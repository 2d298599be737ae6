// bf16 Linear-over-a-sequence on bf16 MFMA (v_mfma_f32_32x32x16_bf16).
//
// Per-sample gradient (appendix "Vectorized Computation", extra dimension
// summed): gW_n[i][j] = s * sum_t B_n[t][i] * A_n[t][j], fp32 accumulation.
// Fused clipped sum: S[i][j] = s * sum_n c_n * sum_t B_n[t][i] * A_n[t][j];
// each sample's product is accumulated on its own and then added with its
// clip factor in fp32, so c_n is never rounded to bf16.
//
// Layout.  MFMA rows run over j (d_in, the weight's contiguous index), MFMA
// columns over i (d_out): each lane ends with four consecutive j of one row
// and stores them as one float4.  Both operands arrive K-major ([t][feature],
// feature contiguous) and are copied into LDS unchanged, 16 bytes at a time.
// The MFMA wants eight consecutive t per lane; gfx950's transposing LDS read
// (ds_read_b64_tr_b16) delivers them: within each 16-lane group, source lane s
// reads four features of row t0 + s/4 and lane i receives feature i of rows
// t0..t0+3.  Two such reads (rows +0 and +4) form one 8-element operand.
// The LDS row stride (320 bytes) puts the four rows of a read on distinct
// banks.
#include "common.hpp"

namespace dpg {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

constexpr int kThreads = 256;
constexpr int TBM = 128;       // j per tile
constexpr int TBN = 128;       // i per tile
constexpr int TBK = 64;        // t per staged chunk
constexpr int RS = 160;        // LDS row stride in bf16 elements (128 features + 32 pad)
constexpr int kCopies = 8;     // 16-byte copies per thread per chunk (both operands)

// One 8-element MFMA operand (eight consecutive t of one feature per lane)
// from a [t][RS] LDS tile: rows t_base.., features f_base..f_base+32.
__device__ __forceinline__ bf16x8_t read_operand(const uint16_t *L, int t_base, int f_base, int lane)
{
    const int g = lane >> 4, s = lane & 15;
    const int t = t_base + 8 * (g >> 1) + (s >> 2);
    const int f = f_base + 16 * (g & 1) + 4 * (s & 3);
    const uint16_t *p = L + t * RS + f;
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)p);
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(p + 4 * RS));
    const i16x8_t v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8_t, v);
}

struct Acc {
    f32x16_t v[2][2];
    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int r = 0; r < 16; ++r) v[x][y][r] = 0.0f;
    }
};

__device__ __forceinline__ void mma_chunk(const uint16_t *As, const uint16_t *Bs, int wm, int wn, int lane,
                                          Acc &acc)
{
#pragma unroll
    for (int ks = 0; ks < TBK / 16; ++ks) {
        bf16x8_t a[2], b[2];
#pragma unroll
        for (int x = 0; x < 2; ++x) a[x] = read_operand(As, 16 * ks, wm + 32 * x, lane);
#pragma unroll
        for (int y = 0; y < 2; ++y) b[y] = read_operand(Bs, 16 * ks, wn + 32 * y, lane);
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
                acc.v[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[x], b[y], acc.v[x][y], 0, 0, 0);
    }
}

// Staging.  Threads 0..127 copy the activation tile (features j), 128..255
// the backprop tile (features i): copy k of thread `slot` is row slot/16 + 8k,
// 16-byte column slot%16.  Rows past T or features past F (F % 8 == 0) read a
// clamped valid address and are zeroed when written.
struct Stage {
    uint4 v[kCopies];
};

struct StageGeom {
    const uint16_t *src;   // operand base of the current sample
    i64 ld;                // row length (features)
    i64 F, f0;             // feature count, first feature of the tile
    uint16_t *L;           // LDS tile
};

__device__ __forceinline__ void stage_load(const StageGeom &sg, i64 T, i64 t0, Stage &st)
{
    const int slot = threadIdx.x & 127;
    const int row0 = slot >> 4, col = slot & 15;
    i64 f = sg.f0 + 8 * col;
    f = f < sg.F ? f : sg.F - 8;
#pragma unroll
    for (int k = 0; k < kCopies; ++k) {
        i64 t = t0 + row0 + 8 * k;
        t = t < T ? t : T - 1;
        st.v[k] = *reinterpret_cast<const uint4 *>(sg.src + t * sg.ld + f);
    }
}

__device__ __forceinline__ void stage_store(const StageGeom &sg, i64 T, i64 t0, const Stage &st)
{
    const int slot = threadIdx.x & 127;
    const int row0 = slot >> 4, col = slot & 15;
    const bool fok = sg.f0 + 8 * col < sg.F;
#pragma unroll
    for (int k = 0; k < kCopies; ++k) {
        const int row = row0 + 8 * k;
        const bool ok = fok && t0 + row < T;
        *reinterpret_cast<uint4 *>(sg.L + row * RS + 8 * col) = ok ? st.v[k] : make_uint4(0u, 0u, 0u, 0u);
    }
}

__device__ __forceinline__ float bias_chunk(const uint16_t *Bs, int feature)
{
    float s = 0.0f;
#pragma unroll 8
    for (int t = 0; t < TBK; ++t) s += bf16_to_f32(Bs[t * RS + feature]);
    return s;
}

__device__ __forceinline__ StageGeom geom_for(const uint16_t *An, const uint16_t *Bn, i64 din, i64 dout, i64 m0,
                                              i64 n0, uint16_t *As, uint16_t *Bs)
{
    const bool isA = threadIdx.x < 128;   // uniform per wave
    StageGeom g;
    g.src = isA ? An : Bn;
    g.ld = isA ? din : dout;
    g.F = g.ld;
    g.f0 = isA ? m0 : n0;
    g.L = isA ? As : Bs;
    return g;
}

// Per-sample gradients.  Block = (sample, j-tile, i-tile).
__global__ __launch_bounds__(kThreads) void bf16_per_sample_kernel(
    const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, i64 T, i64 din, i64 dout, int tiles_m,
    int tiles, float scale, float *__restrict__ gW, float *__restrict__ gb, float *__restrict__ partial)
{
    __shared__ uint16_t As[TBK * RS];
    __shared__ uint16_t Bs[TBK * RS];
    __shared__ float red[16];
    const i64 b = xcd_swizzle(blockIdx.x, gridDim.x);
    const i64 n = b / tiles;
    const int tile = (int)(b % tiles);
    const int tn = tile / tiles_m, tm = tile % tiles_m;     // neighbouring blocks share the i-tile
    const i64 m0 = (i64)tm * TBM, n0 = (i64)tn * TBN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
    const bool do_bias = gb != nullptr && tm == 0;
    const StageGeom sg = geom_for(A + n * T * din, B + n * T * dout, din, dout, m0, n0, As, Bs);

    Acc acc;
    acc.zero();
    float bias_acc = 0.0f;
    const int nchunks = (int)ceil_div(T, TBK);
    // one LDS buffer (several workgroups per CU); the next chunk's loads are in
    // flight in registers while this chunk's MFMAs run
    Stage st;
    stage_load(sg, T, 0, st);
    stage_store(sg, T, 0, st);
    __syncthreads();
    for (int c = 0; c < nchunks; ++c) {
        const bool more = c + 1 < nchunks;
        if (more) stage_load(sg, T, (i64)(c + 1) * TBK, st);
        mma_chunk(As, Bs, wm, wn, lane, acc);
        if (do_bias && tid < TBN) bias_acc += bias_chunk(Bs, tid);
        if (more) {
            __syncthreads();
            stage_store(sg, T, (i64)(c + 1) * TBK, st);
            __syncthreads();
        }
    }

    float sq = 0.0f;
    float *G = gW + n * dout * din;
    const int li = lane & 31, kg = lane >> 5;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const i64 i = n0 + wn + 32 * y + li;
            if (i >= dout) continue;
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const i64 j = m0 + wm + 32 * x + 8 * rb + 4 * kg;
                if (j >= din) continue;   // din % 8 == 0: the four j are all in or all out
                const float g0 = scale * acc.v[x][y][4 * rb + 0], g1 = scale * acc.v[x][y][4 * rb + 1];
                const float g2 = scale * acc.v[x][y][4 * rb + 2], g3 = scale * acc.v[x][y][4 * rb + 3];
                *reinterpret_cast<float4 *>(G + i * din + j) = make_float4(g0, g1, g2, g3);
                sq += g0 * g0 + g1 * g1 + g2 * g2 + g3 * g3;
            }
        }
    if (do_bias && tid < TBN && n0 + tid < dout) {
        const float g = scale * bias_acc;
        gb[n * dout + n0 + tid] = g;
        sq += g * g;
    }
    sq = block_sum(sq, red);
    if (partial && tid == 0) partial[n * tiles + tile] = sq;
}

// Fused clipped sum.  Block = (sample range, j-tile, i-tile); writes the
// range's partial tile (or the final sum when there is one range).
__global__ __launch_bounds__(kThreads) void bf16_clipsum_kernel(
    const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, i64 N, i64 T, i64 din, i64 dout,
    int tiles_m, int tiles, i64 per_split, float scale, const float *__restrict__ norm, float C,
    float *__restrict__ outW, float *__restrict__ outb, i64 strideW, i64 strideb)
{
    __shared__ uint16_t As[TBK * RS];
    __shared__ uint16_t Bs[TBK * RS];
    const i64 bb = xcd_swizzle(blockIdx.x, gridDim.x);
    const int split = (int)(bb / tiles);
    const int tile = (int)(bb % tiles);
    const int tn = tile / tiles_m, tm = tile % tiles_m;
    const i64 m0 = (i64)tm * TBM, n0 = (i64)tn * TBN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
    const i64 s0 = (i64)split * per_split;
    const i64 s1 = s0 + per_split < N ? s0 + per_split : N;
    const bool do_bias = outb != nullptr && tm == 0;

    Acc tot, acc;
    tot.zero();
    acc.zero();
    float bias_tot = 0.0f, bias_acc = 0.0f;
    // (sample, chunk) pairs of this range, flattened so loads run ahead across samples
    // (no 64-bit division in the loop: the sample and chunk advance as counters)
    const int cps = (int)ceil_div(T, TBK);
    const int total = (int)(s1 - s0) * cps;
    const StageGeom sg0 = geom_for(A, B, din, dout, m0, n0, As, Bs);
    const i64 sstride = T * sg0.ld;   // elements between two samples of this thread's operand
    Stage st;
    StageGeom sgn = sg0;
    sgn.src += s0 * sstride;
    if (total > 0) {
        stage_load(sgn, T, 0, st);
        stage_store(sgn, T, 0, st);
    }
    __syncthreads();
    i64 cur_sample = s0;          // sample of chunk c
    int nxt_chunk = 1;            // chunk-in-sample of chunk c + 1
    for (int c = 0; c < total; ++c) {
        const bool more = c + 1 < total;
        const bool sample_done = nxt_chunk == cps;
        if (sample_done) {
            nxt_chunk = 0;
            sgn.src += sstride;
        }
        const i64 tn0 = (i64)nxt_chunk * TBK;
        if (more) stage_load(sgn, T, tn0, st);
        mma_chunk(As, Bs, wm, wn, lane, acc);
        if (do_bias && tid < TBN) bias_acc += bias_chunk(Bs, tid);
        if (sample_done) {
            // the sample's product is complete: add it with its clip factor
            const float cs = scale * clip_factor(norm[cur_sample], C);
            ++cur_sample;
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < 2; ++y)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        tot.v[x][y][r] += cs * acc.v[x][y][r];
                        acc.v[x][y][r] = 0.0f;
                    }
            bias_tot += cs * bias_acc;
            bias_acc = 0.0f;
        }
        if (more) {
            __syncthreads();
            stage_store(sgn, T, tn0, st);
            __syncthreads();
        }
        ++nxt_chunk;
    }

    float *O = outW + (i64)split * strideW;
    const int li = lane & 31, kg = lane >> 5;
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const i64 i = n0 + wn + 32 * y + li;
            if (i >= dout) continue;
#pragma unroll
            for (int rb = 0; rb < 4; ++rb) {
                const i64 j = m0 + wm + 32 * x + 8 * rb + 4 * kg;
                if (j >= din) continue;
                *reinterpret_cast<float4 *>(O + i * din + j) =
                    make_float4(tot.v[x][y][4 * rb + 0], tot.v[x][y][4 * rb + 1], tot.v[x][y][4 * rb + 2],
                                tot.v[x][y][4 * rb + 3]);
            }
        }
    if (do_bias && tid < TBN && n0 + tid < dout) outb[(i64)split * strideb + n0 + tid] = bias_tot;
}

__global__ void bf16_split_sum_kernel(const float *__restrict__ part, int splits, i64 count,
                                      float *__restrict__ out)
{
    const i64 e = (i64)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= count) return;
    out[e] = ordered_sum(part + e, count, splits);
}

}  // namespace

// ---------------------------------------------------------------------------
// host side, called from linear.hip's entry points
// ---------------------------------------------------------------------------
bool bf16_path_ok(const void *A, const void *B, const void *out, i64 T, i64 din, i64 dout)
{
    return T > 1 && din % 8 == 0 && dout % 8 == 0 && aligned(A, 16) && aligned(B, 16) && aligned(out, 16);
}

int bf16_tiles(i64 din, i64 dout) { return (int)(ceil_div(din, TBM) * ceil_div(dout, TBN)); }

void bf16_grad_sample(const void *A, const void *B, i64 N, i64 T, i64 din, i64 dout, float scale, float *gW,
                      float *gb, float *partial, hipStream_t stream)
{
    const int tiles_m = (int)ceil_div(din, TBM);
    const int tiles = bf16_tiles(din, dout);
    bf16_per_sample_kernel<<<(unsigned)(N * tiles), kThreads, 0, stream>>>(
        (const uint16_t *)A, (const uint16_t *)B, T, din, dout, tiles_m, tiles, scale, gW, gb, partial);
}

int bf16_clip_splits(i64 N, i64 T, i64 din, i64 dout)
{
    const int tiles = bf16_tiles(din, dout);
    i64 want = ceil_div(512, tiles);
    if (want > 8) want = 8;         // bound the partial-tile traffic
    if (want > N) want = N;
    if (want < 1) want = 1;
    (void)T;
    const i64 per = ceil_div(N, want);
    return (int)ceil_div(N, per);
}

size_t bf16_clip_workspace(i64 N, i64 T, i64 din, i64 dout)
{
    const int splits = bf16_clip_splits(N, T, din, dout);
    return splits > 1 ? (size_t)splits * (size_t)(din * dout + dout) * sizeof(float) : 0;
}

void bf16_clip_accumulate(const void *A, const void *B, i64 N, i64 T, i64 din, i64 dout, float scale,
                          const float *norm, float C, float *sumW, float *sumb, void *ws, hipStream_t stream)
{
    const int tiles_m = (int)ceil_div(din, TBM);
    const int tiles = bf16_tiles(din, dout);
    const int splits = bf16_clip_splits(N, T, din, dout);
    const i64 per = ceil_div(N, splits);
    const i64 cw = din * dout;
    float *pw = splits > 1 ? (float *)ws : sumW;
    float *pb = sumb ? (splits > 1 ? (float *)ws + (i64)splits * cw : sumb) : nullptr;
    bf16_clipsum_kernel<<<(unsigned)(splits * tiles), kThreads, 0, stream>>>(
        (const uint16_t *)A, (const uint16_t *)B, N, T, din, dout, tiles_m, tiles, per, scale, norm, C, pw, pb,
        cw, dout);
    if (splits > 1) {
        bf16_split_sum_kernel<<<(unsigned)ceil_div(cw, 256), 256, 0, stream>>>(pw, splits, cw, sumW);
        if (sumb) bf16_split_sum_kernel<<<(unsigned)ceil_div(dout, 256), 256, 0, stream>>>(pb, splits, dout, sumb);
    }
}

}  // namespace dpg
