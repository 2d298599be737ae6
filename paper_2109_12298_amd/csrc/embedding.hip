// Embedding per-sample gradients as a deterministic segmented reduction.
//
// Sample n's gradient is non-zero only on the rows of the ids it holds; row v
// is s * sum of B[n][t][:] over its positions t with ids[n][t] = v.  Instead
// of the dense [N][V][D] tensor (which makes embeddings the paper's worst
// case for memory and runtime) the result is CSR over the batch.
//
// Two launches (three when N > 2048):
// Pass 1 (one workgroup per sample): sort the keys (id, t) in LDS.  The keys
//   are unique (t is), so for T <= 512 each key's rank is the number of
//   smaller keys and the sort is one scatter (no barrier per pass); longer
//   samples use a bitonic network.  Equal ids end up in ascending t.  Then
//   the segment index of each sorted position (a prefix count of the "new
//   id" heads), the distinct count and the valid count.
// Pass 2 (G workgroups per sample, G = T / 64 clamped to [1, 8]): the
//   sample's sorted positions are cut into G ranges at segment boundaries
//   (range g starts at the first segment that starts at or after g * P / G),
//   so no segment crosses workgroups.  Each workgroup adds the distinct
//   counts of the samples before n (its first CSR row; a scan launch in
//   between does it for N > 2048), then splits its range over 4 waves.  A
//   wave issues the row loads of 16 positions at once (lanes over columns)
//   and adds them in ascending t, writing every segment that starts and ends
//   in its range; a segment that crosses waves is finished by the wave where
//   it starts, which adds the pieces of the following waves in wave order.
//   So a segment's order is fixed: ascending t within a piece, pieces in t
//   order.  The squared norm is each wave's sum over the rows it wrote, the
//   waves' sums in wave order, then the G workgroups' sums in g order, added
//   by whichever workgroup of the sample finishes last (a per-sample
//   completion counter; no atomics on data, no workgroup waits for another).
#include "common.hpp"

#include <type_traits>

namespace dpg {
namespace {

constexpr int kSortThreads = 1024;
constexpr i64 kMaxT = 4096;
constexpr i64 kRankMaxT = 512;      // rank sort up to here, bitonic beyond
constexpr i64 kPrefixMaxN = 2048;   // pass 2 adds the distinct counts itself up to here
constexpr int kCsrWaves = 4;        // pass 2 workgroup: 256 threads
constexpr int kCsrThreads = 64 * kCsrWaves;
constexpr int kMaxSplit = 8;        // pass 2 workgroups per sample, at most
constexpr int kStage = (int)(kMaxT / kCsrThreads);          // staged positions per thread, at most
constexpr int kPrefixLoads = (int)(kPrefixMaxN / kCsrThreads);
constexpr uint32_t kInvalidHi = 0xffffffffu;   // key high word of an id outside [0, V)

struct EmbWs {
    int32_t *perm;      // [N][T] position t of each sorted position
    int32_t *sidx;      // [N][T] segment index of each sorted position
    int32_t *segid;     // [N][T] id of each segment
    int32_t *counts;    // [N]    distinct valid ids
    int32_t *valid;     // [N]    valid positions
    int32_t *done;      // [N]    pass 2 workgroups of the sample that have finished
    float *sqpart;      // [N][kMaxSplit] squared norm of each pass 2 workgroup's rows
};

// pass 2 workgroups per sample
int split_for(i64 T)
{
    const i64 g = T / 64;
    return (int)(g < 1 ? 1 : (g > kMaxSplit ? kMaxSplit : g));
}

// Exclusive scan of one int per thread over the block (wave scans, then the
// wave totals); returns the total in `total`.  wsum: __shared__ int[16], not
// reused after the call.
__device__ int block_exclusive_scan(int v, int *wsum, int &total)
{
    const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
    const int nw = (int)(blockDim.x / kWave);
    int x = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
    }
    if (lane == kWave - 1) wsum[w] = x;
    lds_barrier();
    int pre = 0, tot = 0;
    for (int i = 0; i < nw; ++i) {
        const int t = wsum[i];
        pre += i < w ? t : 0;
        tot += t;
    }
    total = tot;
    return pre + x - v;
}

__device__ __forceinline__ int pick4(const int (&a)[4], int q)
{
    return q == 0 ? a[0] : q == 1 ? a[1] : q == 2 ? a[2] : a[3];
}

// Rank of each of the T (<= 512) unique keys kk[] among all of them, and
// keys[i] stored at sorted[rank].  Groups of S adjacent lanes own four keys;
// each lane reads every S-th key and compares it with all four (one LDS read
// per four comparisons), then the counts are added over the group.  The
// comparisons bound it (T^2 per sample), hence 32-bit keys where they fit.
template <typename K>
__device__ __forceinline__ void rank_scatter(const K *kk, const uint64_t *keys, uint64_t *sorted, int T, int tid)
{
    const int S = T <= kSortThreads / 4 ? 16 : 8;
    const int grp = tid / S, sub = tid % S;
    K ki[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int i = 4 * grp + q;
        ki[q] = kk[i < T ? i : 0];
    }
    int r[4] = {0, 0, 0, 0};
    int j = sub;
    for (; j + 3 * S < T; j += 4 * S) {
        K kj[4];
#pragma unroll
        for (int a = 0; a < 4; ++a) kj[a] = kk[j + a * S];
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int q = 0; q < 4; ++q) r[q] += kj[a] < ki[q] ? 1 : 0;
    }
    for (; j < T; j += S) {
        const K kj = kk[j];
#pragma unroll
        for (int q = 0; q < 4; ++q) r[q] += kj < ki[q] ? 1 : 0;
    }
    for (int off = S >> 1; off >= 1; off >>= 1)
#pragma unroll
        for (int q = 0; q < 4; ++q) r[q] += __shfl_xor(r[q], off, kWave);
    const int i = 4 * grp + sub;
    if (sub < 4 && i < T) sorted[pick4(r, sub)] = keys[i];
}

__global__ __launch_bounds__(kSortThreads) void emb_sort_kernel(const int64_t *__restrict__ ids, i64 T, i64 V,
                                                                int P2, EmbWs w, int32_t *status)
{
    extern __shared__ uint64_t keys[];           // [2][T] + uint32 [T] (rank sort) or [P2] (bitonic)
    __shared__ int wsum[kSortThreads / kWave];
    const i64 n = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t *idn = ids + n * T;
    const bool rank = T <= kRankMaxT;
    const int L = rank ? (int)T : P2;            // keys in the sorted array
    uint64_t *sorted = rank ? keys + T : keys;
    // 32-bit keys id * T + t (V * T + t for an invalid id) when they fit
    uint32_t *k32 = reinterpret_cast<uint32_t *>(keys + 2 * T);
    const bool small = rank && (uint64_t)(V + 1) * (uint64_t)T <= 0xffffffffull;
    bool bad = false;
    for (int i = tid; i < L; i += kSortThreads) {
        uint64_t k = ~0ull;                      // bitonic padding
        if (i < T) {
            const int64_t id = idn[i];
            const bool ok = id >= 0 && id < V;
            bad |= !ok;
            // an invalid id keeps a unique key that sorts after every valid one
            k = ((uint64_t)(ok ? (uint32_t)id : kInvalidHi) << 32) | (uint32_t)i;
            if (small) k32[i] = (uint32_t)((ok ? id : V) * T + i);
        }
        keys[i] = k;
    }
    if (bad) raise_flag(status, DP_FLAG_BAD_INDEX);
    if (tid == 0) w.done[n] = 0;
    lds_barrier();
    if (rank) {
        if (small) rank_scatter<uint32_t>(k32, keys, sorted, (int)T, tid);
        else rank_scatter<uint64_t>(keys, keys, sorted, (int)T, tid);
        lds_barrier();
    } else {
        for (int k = 2; k <= P2; k <<= 1) {
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int i = tid; i < P2; i += kSortThreads) {
                    const int ixj = i ^ j;
                    if (ixj > i) {
                        const uint64_t a = keys[i], b = keys[ixj];
                        const bool up = (i & k) == 0;
                        if ((a > b) == up) {
                            keys[i] = b;
                            keys[ixj] = a;
                        }
                    }
                }
                lds_barrier();
            }
        }
    }
    // each thread owns a contiguous range of sorted positions: heads of new
    // ids (low half) and valid positions (high half; both at most 4096),
    // counted, then scanned over the block
    const int per = (int)((T + kSortThreads - 1) / kSortThreads);
    const int r0 = tid * per;
    const int r1 = (int)(r0 + per < T ? r0 + per : T);
    int cnt = 0;
    for (int r = r0; r < r1; ++r) {
        const uint32_t hi = (uint32_t)(sorted[r] >> 32);
        if (hi == kInvalidHi) continue;
        cnt += 1 << 16;
        if (r == 0 || (uint32_t)(sorted[r - 1] >> 32) != hi) ++cnt;
    }
    int tot;
    int s = (block_exclusive_scan(cnt, wsum, tot) & 0xffff) - 1;   // segment of the position before r0
    int32_t *perm = w.perm + n * T;
    int32_t *sidx = w.sidx + n * T;
    int32_t *segid = w.segid + n * T;
    for (int r = r0; r < r1; ++r) {
        const uint64_t k = sorted[r];
        const uint32_t hi = (uint32_t)(k >> 32);
        if (hi == kInvalidHi) continue;
        if (r == 0 || (uint32_t)(sorted[r - 1] >> 32) != hi) segid[++s] = (int32_t)hi;
        perm[r] = (int32_t)(k & 0xffffffffu);
        sidx[r] = s;
    }
    if (tid == 0) {
        w.counts[n] = tot & 0xffff;
        w.valid[n] = tot >> 16;
    }
}

// row_ptr[n + 1] = the distinct counts of samples 0..n (one workgroup; the
// path for more samples than pass 2 adds up itself)
__global__ __launch_bounds__(256) void emb_scan_kernel(const int32_t *__restrict__ counts, i64 N,
                                                       int64_t *__restrict__ row_ptr)
{
    __shared__ int64_t buf[256];
    __shared__ int64_t carry;
    const int tid = threadIdx.x;
    if (tid == 0) {
        carry = 0;
        row_ptr[0] = 0;
    }
    __syncthreads();
    for (i64 c = 0; c < N; c += 256) {
        const i64 n = c + tid;
        const int64_t v = n < N ? counts[n] : 0;
        buf[tid] = v;
        __syncthreads();
        for (int off = 1; off < 256; off <<= 1) {
            const int64_t x = tid >= off ? buf[tid - off] : 0;
            __syncthreads();
            buf[tid] += x;
            __syncthreads();
        }
        if (n < N) row_ptr[n + 1] = carry + buf[tid];
        __syncthreads();
        if (tid == 0) carry += buf[255];
        __syncthreads();
    }
}

// VEC consecutive row elements as floats (VEC = 4: one 16-byte fp32 or
// 8-byte bf16 load, the address aligned to that size).
template <typename T, int VEC>
__device__ __forceinline__ void load_vec(const T *p, float (&v)[VEC])
{
    if constexpr (VEC == 4 && std::is_same<T, float>::value) {
        const float4 q = *reinterpret_cast<const float4 *>(p);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
    } else if constexpr (VEC == 4) {
        const uint2 q = *reinterpret_cast<const uint2 *>(p);
        v[0] = bf16_to_f32((uint16_t)(q.x & 0xffffu)); v[1] = bf16_to_f32((uint16_t)(q.x >> 16));
        v[2] = bf16_to_f32((uint16_t)(q.y & 0xffffu)); v[3] = bf16_to_f32((uint16_t)(q.y >> 16));
    } else {
#pragma unroll
        for (int i = 0; i < VEC; ++i) v[i] = load_elem<T>(p, i);
    }
}

constexpr int kBatch = 16;    // positions whose row loads a wave has in flight together

// pieces of segments that cross waves, per wave: the end of a segment that
// started in an earlier wave (head), the start of one that continues (tail),
// or the middle of one that covers the whole range (mid)
enum { kHead = 0, kTail = 1, kMid = 2 };

// The walk of the sorted positions [lo, hi) by WAVES waves: wave wv takes a
// contiguous share, adds each segment's rows in ascending t (rows of Bn, the
// sample's backprops) and writes s * sum as CSR row base + segment; a segment
// that crosses waves is finished by the wave where it starts, which adds the
// following waves' pieces in wave order.  sq accumulates the squares of the
// rows this thread wrote.  Every thread of the workgroup calls it (it holds
// workgroup barriers).
template <typename T, int VEC, int WAVES>
__device__ __forceinline__ void walk_rows(const T *__restrict__ Bn, i64 D, float scale,
                                          const int32_t *perm, const int32_t *sidx, int P, int lo, int hi,
                                          i64 base, float *__restrict__ rows, i64 cap,
                                          float (*piece)[3][64 * VEC], int (*pseg)[3], int wv, int lane, float &sq)
{
    constexpr int CB = 64 * VEC;                         // columns per column block
    const int R = (hi - lo + WAVES - 1) / WAVES;       // sorted positions per wave
    const int r_lo = lo + wv * R < hi ? lo + wv * R : hi;
    const int r_hi = r_lo + R < hi ? r_lo + R : hi;
    // does the wave's first segment start before its range, its last continue after it?
    const bool first_cont = r_lo < r_hi && r_lo > lo && sidx[r_lo - 1] == sidx[r_lo];
    const bool last_cont = r_lo < r_hi && r_hi < hi && sidx[r_hi] == sidx[r_hi - 1];

    auto finish = [&](i64 s, const float (&acc)[VEC], i64 c, bool on) {
        const i64 k = base + s;
        if (on) {
            float gr[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                gr[i] = scale * acc[i];
                sq += gr[i] * gr[i];
            }
            if (k < cap) {
                if constexpr (VEC == 4)
                    *reinterpret_cast<float4 *>(rows + k * D + c) = make_float4(gr[0], gr[1], gr[2], gr[3]);
                else
                    rows[k * D + c] = gr[0];
            }
        }
    };

    for (i64 c0c = 0; c0c < D; c0c += CB) {
        const i64 c = c0c + (i64)VEC * lane;
        const bool on = c < D;
        const i64 cc = on ? c : 0;
        float acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0f;
        bool started_here = !first_cont;
        if (lane < 3) pseg[wv][lane] = -1;
        for (int r0 = r_lo; r0 < r_hi; r0 += kBatch) {
            // lane l (and l + 16, l + 32, l + 48) holds position r0 + l of the
            // batch: its t, its segment, whether the segment ends there
            const int rl = r0 + (lane & (kBatch - 1));
            const bool in = rl < r_hi;
            const int tl = perm[in ? rl : r0];
            const int sl = sidx[in ? rl : r0];
            const bool ends = in && (rl + 1 == P || sidx[rl + 1] != sl);
            const uint32_t endm = (uint32_t)__ballot(ends);
            float v[kBatch][VEC];
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                const int t = __builtin_amdgcn_readlane(tl, j);
                load_vec<T, VEC>(Bn + (i64)t * D + cc, v[j]);
            }
            // (fully unrolled with a uniform guard instead of a break, so
            // that v stays in registers)
#pragma unroll
            for (int j = 0; j < kBatch; ++j) {
                if (r0 + j >= r_hi) continue;
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += v[j][i];
                if ((endm >> j) & 1u) {
                    const int s = __builtin_amdgcn_readlane(sl, j);
                    if (started_here) {
                        finish(s, acc, c, on);
                    } else {
                        // the end of a segment from an earlier wave
#pragma unroll
                        for (int i = 0; i < VEC; ++i) piece[wv][kHead][VEC * lane + i] = acc[i];
                        if (lane == 0) pseg[wv][kHead] = s;
                    }
#pragma unroll
                    for (int i = 0; i < VEC; ++i) acc[i] = 0.0f;
                    started_here = true;
                }
            }
        }
        if (last_cont) {
            const int kind = started_here ? kTail : kMid;
#pragma unroll
            for (int i = 0; i < VEC; ++i) piece[wv][kind][VEC * lane + i] = acc[i];
            if (lane == 0) pseg[wv][kind] = sidx[r_hi - 1];
        }
        lds_barrier();
        // a segment that starts in this wave and continues: add the following
        // waves' pieces in wave order, then write it
        if (pseg[wv][kTail] >= 0) {
            const int s = pseg[wv][kTail];
#pragma unroll
            for (int i = 0; i < VEC; ++i) acc[i] = piece[wv][kTail][VEC * lane + i];
            for (int x = wv + 1; x < WAVES; ++x) {
                if (pseg[x][kMid] == s) {
#pragma unroll
                    for (int i = 0; i < VEC; ++i) acc[i] += piece[x][kMid][VEC * lane + i];
                } else {
#pragma unroll
                    for (int i = 0; i < VEC; ++i) acc[i] += piece[x][kHead][VEC * lane + i];
                    break;
                }
            }
            finish(s, acc, c, on);
        }
        lds_barrier();                                   // the pieces are rewritten by the next block
    }

}

template <typename T, int VEC>
__global__ __launch_bounds__(kCsrThreads) void emb_csr_kernel(
    const T *__restrict__ B, i64 Tn, i64 D, float scale, EmbWs w, int G, int prefix_here,
    int64_t *__restrict__ row_ptr, int64_t *__restrict__ uniq, float *__restrict__ rows, i64 cap,
    float *__restrict__ sqnorm, int32_t *status)
{
    constexpr int CB = 64 * VEC;                         // columns per column block
    extern __shared__ int32_t order[];                   // the sample's perm, sidx, segid (3 * Tn)
    __shared__ float piece[kCsrWaves][3][CB];
    __shared__ int pseg[kCsrWaves][3];                   // segment of each piece, -1 for none
    __shared__ float wsq[kCsrWaves];
    __shared__ int64_t wpart[kCsrWaves];
    __shared__ int wbound[kCsrWaves][2];
    const i64 n = blockIdx.x / G;
    const int g = (int)(blockIdx.x % G);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int u = w.counts[n], P = w.valid[n];

    // Every load that does not depend on another is issued before the first
    // wait: the distinct counts of the samples before n (N <= 2048) and the
    // sample's sorted positions, segments and ids (T <= 4096).  Bounded
    // raw-buffer loads read zero past the end.
    const __amdgpu_buffer_rsrc_t rcnt = sample_rsrc(w.counts, prefix_here ? (uint32_t)n * 4u : 0u);
    const __amdgpu_buffer_rsrc_t rperm = sample_rsrc(w.perm + n * Tn, (uint32_t)P * 4u);
    const __amdgpu_buffer_rsrc_t rsidx = sample_rsrc(w.sidx + n * Tn, (uint32_t)P * 4u);
    const __amdgpu_buffer_rsrc_t rseg = sample_rsrc(w.segid + n * Tn, (uint32_t)u * 4u);
    int64_t part = 0, base_in = 0;
    int32_t cl[kPrefixLoads];
#pragma unroll
    for (int k = 0; k < kPrefixLoads; ++k) cl[k] = buffer_load_i32(rcnt, 4u * (uint32_t)(tid + kCsrThreads * k));
    if (!prefix_here) base_in = row_ptr[n];
    int32_t pv[kStage], sv[kStage], gv[kStage];
#pragma unroll
    for (int k = 0; k < kStage; ++k) {
        pv[k] = sv[k] = gv[k] = 0;
        if (kCsrThreads * k < P) {
            const uint32_t o = 4u * (uint32_t)(tid + kCsrThreads * k);
            pv[k] = buffer_load_i32(rperm, o);
            sv[k] = buffer_load_i32(rsidx, o);
            gv[k] = buffer_load_i32(rseg, o);
        }
    }
    int32_t *perm = order;
    int32_t *sidx = order + Tn;
    int32_t *segid = order + 2 * Tn;
#pragma unroll
    for (int k = 0; k < kStage; ++k) {
        const int r = tid + kCsrThreads * k;
        if (r < P) {
            perm[r] = pv[k];
            sidx[r] = sv[k];
            segid[r] = gv[k];    // u <= P, so every segment is staged
        }
    }
#pragma unroll
    for (int k = 0; k < kPrefixLoads; ++k) part += cl[k];
    for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, kWave);
    if (lane == 0) wpart[wv] = part;
    lds_barrier();

    // the workgroup's range [lo, hi): from the first segment start at or after
    // g * P / G to the first at or after (g + 1) * P / G
    // (the lowest lane of a ballot is the wave's first such position, then
    // the minimum over the waves)
    const int c0 = (int)((uint32_t)(g * P) / (uint32_t)G), c1 = (int)((uint32_t)((g + 1) * P) / (uint32_t)G);
    int f0 = P, f1 = P;
    for (int rb = wv * 64; rb < P; rb += kCsrThreads) {
        const int r = rb + lane;
        const bool start = r < P && (r == 0 || sidx[r] != sidx[r - 1]);
        const uint64_t b0 = __ballot(start && r >= c0), b1 = __ballot(start && r >= c1);
        if (b0 && f0 == P) f0 = rb + __ffsll((unsigned long long)b0) - 1;
        if (b1 && f1 == P) f1 = rb + __ffsll((unsigned long long)b1) - 1;
    }
    if (lane == 0) {
        wbound[wv][0] = f0;
        wbound[wv][1] = f1;
    }
    i64 base = base_in;
    if (prefix_here) {
        base = 0;
        for (int i = 0; i < kCsrWaves; ++i) base += wpart[i];
    }
    lds_barrier();
    int lo = P, hi = P;
    for (int i = 0; i < kCsrWaves; ++i) {
        lo = wbound[i][0] < lo ? wbound[i][0] : lo;
        hi = wbound[i][1] < hi ? wbound[i][1] : hi;
    }

    const T *Bn = B + n * Tn * D;
    float sq = 0.0f;
    walk_rows<T, VEC, kCsrWaves>(Bn, D, scale, perm, sidx, P, lo, hi, base, rows, cap, piece, pseg, wv, lane, sq);

    // the ids of the segments the workgroup owns and the sample's CSR bound,
    // stored last (a store issued before the walk would make the walk's first
    // loads wait for it)
    if (lo < hi) {
        const int s_first = sidx[lo], s_last = sidx[hi - 1];
        for (int s = s_first + tid; s <= s_last; s += kCsrThreads)
            if (base + s < cap) uniq[base + s] = segid[s];
    }
    if (g == 0 && tid == 0) {
        if (prefix_here) {
            row_ptr[n + 1] = base + u;
            if (n == 0) row_ptr[0] = 0;
        }
        if (base + u > cap) raise_flag(status, DP_FLAG_CAP);
    }
    if (!sqnorm) return;
    sq = wave_sum(sq);
    if (lane == 0) wsq[wv] = sq;
    lds_barrier();
    if (tid != 0) return;
    float t = 0.0f;
    for (int i = 0; i < kCsrWaves; ++i) t += wsq[i];
    if (G == 1) {
        sqnorm[n] = t;
        return;
    }
    // The sample's last workgroup to finish adds the G sums in g order.  The
    // sum is stored with device-scope coherence (written through to where
    // every XCD sees it) and acknowledged before the counter is bumped; the
    // last workgroup reads the sums the same way after its bump returns.
    // (An acquire-release counter would also write back every dirty line of
    // the XCD's L2, the rows included, for each workgroup.)
    __hip_atomic_store(w.sqpart + n * kMaxSplit + g, t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const int before = __hip_atomic_fetch_add(w.done + n, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (before != G - 1) return;
    float tot = 0.0f;
    for (int x = 0; x < G; ++x)
        tot += __hip_atomic_load(w.sqpart + n * kMaxSplit + x, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    sqnorm[n] = tot;
}

// ---------------------------------------------------------------------------
// One launch for T <= 512 (after a fill that clears the ticket and the
// per-sample states): one workgroup of 16 waves per sample sorts, walks and
// writes the sample's CSR block.  The sample's first CSR row (the distinct
// counts of the samples before it) comes from a decoupled look-back: each
// workgroup publishes its distinct count as soon as its sort is done, then
// adds its predecessors' published values, 64 at a time, back to the nearest
// one that already holds its inclusive prefix, and publishes its own
// inclusive prefix.  Samples are taken in ticket order (an atomic counter),
// so a workgroup only waits for samples whose workgroups already run; the
// wait is bounded (past the bound it sets DP_FLAG_WAIT and counts the
// missing sample as empty).  The sums are those of the two-launch path's
// walk over 16 waves: same segments, same ascending-t order within a piece.
// ---------------------------------------------------------------------------
constexpr int kFusedWaves = 16;
constexpr int kFusedThreads = 64 * kFusedWaves;
constexpr uint64_t kAgg = 1ull << 62;          // state: the sample's distinct count
constexpr uint64_t kIncl = 2ull << 62;         // state: its inclusive prefix
constexpr uint64_t kStateVal = (1ull << 62) - 1;
constexpr int kSpinMax = 1 << 20;

template <typename T, int VEC>
__global__ __launch_bounds__(kFusedThreads) void emb_fused_kernel(
    const int64_t *__restrict__ ids, const T *__restrict__ B, i64 Tn, i64 V, i64 D, float scale,
    int32_t *__restrict__ ticket, uint64_t *__restrict__ state, int64_t *__restrict__ row_ptr,
    int64_t *__restrict__ uniq, float *__restrict__ rows, i64 cap, float *__restrict__ sqnorm, int32_t *status)
{
    constexpr int CB = 64 * VEC;
    extern __shared__ uint64_t keys[];           // keys [T], sorted [T], 32-bit keys [T], perm, sidx, segid [T] each
    __shared__ float piece[kFusedWaves][3][CB];
    __shared__ int pseg[kFusedWaves][3];
    __shared__ float wsq[kFusedWaves];
    __shared__ int wsum[kFusedWaves];
    __shared__ int s_n;
    __shared__ int64_t s_base;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    if (tid == 0) s_n = __hip_atomic_fetch_add(ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    const i64 n = s_n;
    const int Tp = (int)Tn;
    const int64_t *idn = ids + n * Tn;
    uint64_t *sorted = keys + Tp;
    uint32_t *k32 = reinterpret_cast<uint32_t *>(keys + 2 * Tp);
    int32_t *perm = reinterpret_cast<int32_t *>(k32 + Tp);
    int32_t *sidx = perm + Tp;
    int32_t *segid = sidx + Tp;

    // the keys (id, t), unique; 32-bit when they fit; an invalid id sorts last
    const bool small = (uint64_t)(V + 1) * (uint64_t)Tn <= 0xffffffffull;
    bool bad = false;
    for (int i = tid; i < Tp; i += kFusedThreads) {
        const int64_t id = idn[i];
        const bool ok = id >= 0 && id < V;
        bad |= !ok;
        keys[i] = ((uint64_t)(ok ? (uint32_t)id : kInvalidHi) << 32) | (uint32_t)i;
        if (small) k32[i] = (uint32_t)((ok ? id : V) * Tn + i);
    }
    if (bad) raise_flag(status, DP_FLAG_BAD_INDEX);
    lds_barrier();
    if (small) rank_scatter<uint32_t>(k32, keys, sorted, Tp, tid);
    else rank_scatter<uint64_t>(keys, keys, sorted, Tp, tid);
    lds_barrier();
    // heads of new ids and valid positions per thread (at most one position
    // each here), scanned over the workgroup
    int cnt = 0;
    if (tid < Tp) {
        const uint32_t hi = (uint32_t)(sorted[tid] >> 32);
        if (hi != kInvalidHi) {
            cnt = 1 << 16;
            if (tid == 0 || (uint32_t)(sorted[tid - 1] >> 32) != hi) ++cnt;
        }
    }
    int tot;
    const int sx = (block_exclusive_scan(cnt, wsum, tot) & 0xffff) - 1;
    if (tid < Tp) {
        const uint64_t k = sorted[tid];
        const uint32_t hi = (uint32_t)(k >> 32);
        if (hi != kInvalidHi) {
            const bool head = tid == 0 || (uint32_t)(sorted[tid - 1] >> 32) != hi;
            const int s = head ? sx + 1 : sx;
            if (head) segid[s] = (int32_t)hi;
            perm[tid] = (int32_t)(k & 0xffffffffu);
            sidx[tid] = s;
        }
    }
    const int u = tot & 0xffff, P = tot >> 16;

    // the first CSR row of the sample
    if (wv == 0) {
        if (lane == 0)
            __hip_atomic_store(state + n, (n == 0 ? kIncl : kAgg) | (uint64_t)u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        int64_t excl = 0;
        bool timed_out = false;
        for (i64 j = n - 1; j >= 0; j -= kWave) {
            const i64 jj = j - lane;
            uint64_t v = kIncl;                        // lanes past sample 0 add nothing
            if (jj >= 0) {
                int spins = 0;
                v = __hip_atomic_load(state + jj, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                while ((v >> 62) == 0 && spins < kSpinMax) {
                    __builtin_amdgcn_s_sleep(1);
                    v = __hip_atomic_load(state + jj, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    ++spins;
                }
                timed_out |= (v >> 62) == 0;
            }
            // the nearest predecessor holding an inclusive prefix ends the look-back
            const uint64_t incl = __ballot(jj >= 0 && (v >> 62) == 2);
            const int stop = incl ? __ffsll((unsigned long long)incl) - 1 : kWave;
            int64_t x = (jj >= 0 && lane <= stop) ? (int64_t)(v & kStateVal) : 0;
            for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, kWave);
            excl += x;
            if (incl) break;
        }
        if (__ballot(timed_out) && lane == 0) raise_flag(status, DP_FLAG_WAIT);
        if (lane == 0) {
            if (n > 0)
                __hip_atomic_store(state + n, kIncl | (uint64_t)(excl + u), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            s_base = excl;
        }
    }
    __syncthreads();
    const i64 base = s_base;

    float sq = 0.0f;
    walk_rows<T, VEC, kFusedWaves>(B + n * Tn * D, D, scale, perm, sidx, P, 0, P, base, rows, cap, piece, pseg,
                                   wv, lane, sq);
    for (int s = tid; s < u; s += kFusedThreads)
        if (base + s < cap) uniq[base + s] = segid[s];
    if (tid == 0) {
        row_ptr[n + 1] = base + u;
        if (n == 0) row_ptr[0] = 0;
        if (base + u > cap) raise_flag(status, DP_FLAG_CAP);
    }
    if (!sqnorm) return;
    sq = wave_sum(sq);
    if (lane == 0) wsq[wv] = sq;
    lds_barrier();
    if (tid == 0) {
        float t = 0.0f;
        for (int i = 0; i < kFusedWaves; ++i) t += wsq[i];
        sqnorm[n] = t;
    }
}

EmbWs carve(void *ws, i64 N, i64 T)
{
    EmbWs w;
    char *p = (char *)ws;
    w.perm = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N * T, 256);
    w.sidx = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N * T, 256);
    w.segid = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N * T, 256);
    w.counts = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N, 256);
    w.valid = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N, 256);
    w.done = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N, 256);
    w.sqpart = (float *)p;
    return w;
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_grad_sample_embedding_workspace_bytes(int64_t N, int64_t T)
{
    if (N <= 0 || T < 0) return 0;
    return 3 * align_up(sizeof(int32_t) * N * T, 256) + 3 * align_up(sizeof(int32_t) * N, 256) +
           align_up(sizeof(float) * N * kMaxSplit, 256);
}

extern "C" dp_status dp_grad_sample_embedding(const int64_t *ids, const void *B, dp_dtype dt,
                                              int64_t N, int64_t T, int64_t V, int64_t D,
                                              float scale, int64_t *row_ptr, int64_t *uniq_ids,
                                              float *rows, int64_t cap, float *sqnorm,
                                              int32_t *status, void *ws, size_t ws_bytes,
                                              hipStream_t stream)
{
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && T >= 0 && V >= 1 && D >= 1 && cap >= 0, DP_EINVAL);
    DPG_REQUIRE(V < (i64(1) << 31), DP_EINVAL);
    DPG_REQUIRE(T <= kMaxT, DP_EUNSUPPORTED);
    // 32-bit sorted-position indices, and one pass 2 workgroup per sample and range
    DPG_REQUIRE(N * T < (i64(1) << 31) && N * kMaxSplit < (i64(1) << 31), DP_EUNSUPPORTED);
    DPG_REQUIRE(row_ptr != nullptr, DP_EINVAL);
    DPG_REQUIRE(N * T == 0 || (ids != nullptr && B != nullptr), DP_EINVAL);
    DPG_REQUIRE(cap == 0 || (uniq_ids != nullptr && rows != nullptr), DP_EINVAL);
    const size_t need = dp_grad_sample_embedding_workspace_bytes(N, T);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) {
        // row_ptr[0] = 0 for an empty batch
        emb_scan_kernel<<<1, 256, 0, stream>>>(nullptr, 0, row_ptr);
        return launch_status();
    }
    // four columns per lane when every row starts on a 16-byte (fp32) or
    // 8-byte (bf16) boundary, and rows likewise
    const bool vec = D % 4 == 0 && aligned(rows, 16) && aligned(B, dt == DP_F32 ? 16 : 8);
    if (T > 0 && T <= kRankMaxT) {
        // one launch after clearing the ticket and the N per-sample states
        int32_t *ticket = (int32_t *)ws;
        uint64_t *state = (uint64_t *)((char *)ws + 256);
        zero_fill((float *)ws, (i64)((256 + 8 * (size_t)N) / 4), stream);
        const size_t flds = 32 * (size_t)T;
        if (dt == DP_F32) {
            if (vec)
                emb_fused_kernel<float, 4><<<(unsigned)N, kFusedThreads, flds, stream>>>(
                    ids, (const float *)B, T, V, D, scale, ticket, state, row_ptr, uniq_ids, rows, cap, sqnorm, status);
            else
                emb_fused_kernel<float, 1><<<(unsigned)N, kFusedThreads, flds, stream>>>(
                    ids, (const float *)B, T, V, D, scale, ticket, state, row_ptr, uniq_ids, rows, cap, sqnorm, status);
        } else {
            if (vec)
                emb_fused_kernel<uint16_t, 4><<<(unsigned)N, kFusedThreads, flds, stream>>>(
                    ids, (const uint16_t *)B, T, V, D, scale, ticket, state, row_ptr, uniq_ids, rows, cap, sqnorm,
                    status);
            else
                emb_fused_kernel<uint16_t, 1><<<(unsigned)N, kFusedThreads, flds, stream>>>(
                    ids, (const uint16_t *)B, T, V, D, scale, ticket, state, row_ptr, uniq_ids, rows, cap, sqnorm,
                    status);
        }
        return launch_status();
    }
    EmbWs w = carve(ws, N, T);
    int P2 = 1;
    while (P2 < T) P2 <<= 1;
    const size_t lds = T <= kRankMaxT ? (2 * sizeof(uint64_t) + sizeof(uint32_t)) * (size_t)(T > 0 ? T : 1)
                                      : sizeof(uint64_t) * P2;
    emb_sort_kernel<<<(unsigned)N, kSortThreads, lds, stream>>>(ids, T, V, P2, w, status);
    const int prefix_here = N <= kPrefixMaxN ? 1 : 0;
    if (!prefix_here) emb_scan_kernel<<<1, 256, 0, stream>>>(w.counts, N, row_ptr);
    const int G = split_for(T);
    const unsigned grid = (unsigned)(N * G);
    const size_t olds = 3 * sizeof(int32_t) * (size_t)(T > 0 ? T : 1);
    if (dt == DP_F32) {
        if (vec)
            emb_csr_kernel<float, 4><<<grid, kCsrThreads, olds, stream>>>((const float *)B, T, D, scale, w, G,
                                                                          prefix_here, row_ptr, uniq_ids, rows,
                                                                          cap, sqnorm, status);
        else
            emb_csr_kernel<float, 1><<<grid, kCsrThreads, olds, stream>>>((const float *)B, T, D, scale, w, G,
                                                                          prefix_here, row_ptr, uniq_ids, rows,
                                                                          cap, sqnorm, status);
    } else {
        if (vec)
            emb_csr_kernel<uint16_t, 4><<<grid, kCsrThreads, olds, stream>>>((const uint16_t *)B, T, D, scale, w,
                                                                             G, prefix_here, row_ptr, uniq_ids,
                                                                             rows, cap, sqnorm, status);
        else
            emb_csr_kernel<uint16_t, 1><<<grid, kCsrThreads, olds, stream>>>((const uint16_t *)B, T, D, scale, w,
                                                                             G, prefix_here, row_ptr, uniq_ids,
                                                                             rows, cap, sqnorm, status);
    }
    return launch_status();
}
