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
// feature contiguous) while the MFMA wants eight consecutive t per lane, so
// staging loads 8x8 blocks (eight 16-byte rows of eight features), transposes
// them in registers and writes eight 16-byte LDS rows with t contiguous.
// LDS rows are padded by 16 bytes so the 16-byte operand reads of 16 lanes hit
// distinct banks.
#include "common.hpp"

namespace dpg {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int TBM = 128;      // j per tile
constexpr int TBN = 128;      // i per tile
constexpr int TBK = 64;       // t per staged chunk
constexpr int LDK = TBK + 8;  // LDS row stride in bf16 elements

__device__ __forceinline__ uint32_t lo_pair(uint32_t a, uint32_t b) { return (a & 0xffffu) | (b << 16); }
__device__ __forceinline__ uint32_t hi_pair(uint32_t a, uint32_t b) { return (a >> 16) | (b & 0xffff0000u); }

// One operand chunk: rows t0..t0+TBK of a [T][ld] bf16 matrix, features
// f0..f0+128.  Thread `slot` (0..127) owns the 8x8 block (t-block slot/16,
// feature-block slot%16): load_8x8 fetches its eight 16-byte rows into
// registers, store_8x8 transposes them and writes L[feature][t] (row stride
// LDK).  Splitting the two lets the next chunk's loads fly during the MFMAs.
struct Block8 {
    uint4 r[8];
};

__device__ __forceinline__ void load_8x8(const uint16_t *__restrict__ src, i64 ld, i64 T, i64 t0, i64 F, i64 f0,
                                         int slot, Block8 &in)
{
    const int tb = slot >> 4, fb = slot & 15;
    const i64 f = f0 + 8 * fb;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
        const i64 t = t0 + 8 * tb + r;
        if (t < T && f < F) in.r[r] = *reinterpret_cast<const uint4 *>(src + t * ld + f);
        else in.r[r] = make_uint4(0u, 0u, 0u, 0u);
    }
}

__device__ __forceinline__ void store_8x8(const Block8 &in, int slot, uint16_t *L)
{
    const int tb = slot >> 4, fb = slot & 15;
    // out[q] = the eight t-values of feature f+q, pairs (t=2w, 2w+1) per word
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        uint32_t w[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            const uint32_t *a = reinterpret_cast<const uint32_t *>(&in.r[2 * p]);
            const uint32_t *b = reinterpret_cast<const uint32_t *>(&in.r[2 * p + 1]);
            w[p] = (q & 1) ? hi_pair(a[q >> 1], b[q >> 1]) : lo_pair(a[q >> 1], b[q >> 1]);
        }
        *reinterpret_cast<uint4 *>(L + (8 * fb + q) * LDK + 8 * tb) = make_uint4(w[0], w[1], w[2], w[3]);
    }
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
    const int li = lane & 31, kg = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < TBK / 16; ++ks) {
        bf16x8_t a[2], b[2];
#pragma unroll
        for (int x = 0; x < 2; ++x)
            a[x] = *reinterpret_cast<const bf16x8_t *>(As + (wm + 32 * x + li) * LDK + 16 * ks + 8 * kg);
#pragma unroll
        for (int y = 0; y < 2; ++y)
            b[y] = *reinterpret_cast<const bf16x8_t *>(Bs + (wn + 32 * y + li) * LDK + 16 * ks + 8 * kg);
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
                acc.v[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[x], b[y], acc.v[x][y], 0, 0, 0);
    }
}

// Threads 0..127 stage the activation operand (features j), 128..255 the
// backprop operand (features i).
__device__ __forceinline__ void load_chunk(const uint16_t *An, const uint16_t *Bn, i64 T, i64 t0, i64 din,
                                           i64 dout, i64 m0, i64 n0, Block8 &in)
{
    const int tid = threadIdx.x;
    if (tid < 128) load_8x8(An, din, T, t0, din, m0, tid, in);
    else load_8x8(Bn, dout, T, t0, dout, n0, tid - 128, in);
}

__device__ __forceinline__ void store_chunk(const Block8 &in, uint16_t *As, uint16_t *Bs)
{
    const int tid = threadIdx.x;
    if (tid < 128) store_8x8(in, tid, As);
    else store_8x8(in, tid - 128, Bs);
}

__device__ __forceinline__ float bias_chunk(const uint16_t *Bs, int row)
{
    float s = 0.0f;
#pragma unroll 8
    for (int t = 0; t < TBK; ++t) s += bf16_to_f32(Bs[row * LDK + t]);
    return s;
}

// Per-sample gradients.  Block = (sample, j-tile, i-tile).
__global__ __launch_bounds__(kThreads) void bf16_per_sample_kernel(
    const uint16_t *__restrict__ A, const uint16_t *__restrict__ B, i64 T, i64 din, i64 dout, int tiles_m,
    int tiles, float scale, float *__restrict__ gW, float *__restrict__ gb, float *__restrict__ partial)
{
    __shared__ uint16_t As[TBM * LDK];
    __shared__ uint16_t Bs[TBN * LDK];
    __shared__ float red[16];
    const i64 b = xcd_swizzle(blockIdx.x, gridDim.x);
    const i64 n = b / tiles;
    const int tile = (int)(b % tiles);
    const int tn = tile / tiles_m, tm = tile % tiles_m;     // neighbouring blocks share the i-tile
    const i64 m0 = (i64)tm * TBM, n0 = (i64)tn * TBN;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;
    const uint16_t *An = A + n * T * din;
    const uint16_t *Bn = B + n * T * dout;
    const bool do_bias = gb != nullptr && tm == 0;

    Acc acc;
    acc.zero();
    float bias_acc = 0.0f;
    const int nchunks = (int)ceil_div(T, TBK);
    // one LDS buffer (four workgroups fit a CU); the next chunk's global loads
    // are in flight in registers while this chunk's MFMAs run
    Block8 in;
    load_chunk(An, Bn, T, 0, din, dout, m0, n0, in);
    store_chunk(in, As, Bs);
    __syncthreads();
    for (int c = 0; c < nchunks; ++c) {
        const bool more = c + 1 < nchunks;
        if (more) load_chunk(An, Bn, T, (i64)(c + 1) * TBK, din, dout, m0, n0, in);
        mma_chunk(As, Bs, wm, wn, lane, acc);
        if (do_bias && tid < TBN) bias_acc += bias_chunk(Bs, tid);
        if (more) {
            __syncthreads();
            store_chunk(in, As, Bs);
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
    __shared__ uint16_t As[TBM * LDK];
    __shared__ uint16_t Bs[TBN * LDK];
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
    const int cps = (int)ceil_div(T, TBK);
    const i64 total = (s1 - s0) * cps;
    Block8 in;
    if (total > 0) {
        load_chunk(A + s0 * T * din, B + s0 * T * dout, T, 0, din, dout, m0, n0, in);
        store_chunk(in, As, Bs);
    }
    __syncthreads();
    for (i64 c = 0; c < total; ++c) {
        const bool more = c + 1 < total;
        if (more) {
            const i64 nn = s0 + (c + 1) / cps;
            const i64 t0 = (i64)((c + 1) % cps) * TBK;
            load_chunk(A + nn * T * din, B + nn * T * dout, T, t0, din, dout, m0, n0, in);
        }
        mma_chunk(As, Bs, wm, wn, lane, acc);
        if (do_bias && tid < TBN) bias_acc += bias_chunk(Bs, tid);
        if ((c + 1) % cps == 0) {
            // the sample's product is complete: add it with its clip factor
            const float cs = scale * clip_factor(norm[s0 + c / cps], C);
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
            store_chunk(in, As, Bs);
            __syncthreads();
        }
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
