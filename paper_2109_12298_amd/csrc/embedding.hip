// Embedding per-sample gradients as a deterministic segmented reduction.
//
// Sample n's gradient is non-zero only on the rows of the ids it holds; row v
// is s * sum of B[n][t][:] over its positions t with ids[n][t] = v.  Instead
// of the dense [N][V][D] tensor (which makes embeddings the paper's worst
// case for memory and runtime) the result is CSR over the batch.
//
// Pass 1 (one workgroup per sample): bitonic sort of the keys (id, t) in LDS;
//   since t is unique the order is total, so equal ids stay in ascending t.
//   Segment starts come from a block scan of the "new id" flags.
// Pass 2 (one workgroup): exclusive scan of the per-sample distinct counts
//   into row_ptr.
// Pass 3 (one wave per sample and segment slot, so the grid fills the chip
//   even for a small batch): the wave sums the segment's backprop rows in
//   ascending t, eight positions' loads in flight at a time (32 for segments
//   longer than eight, such as a hot id's), lanes over the
//   columns (four per lane when the rows allow 16- or 8-byte loads), and
//   writes the CSR row and its squared norm; the sample's norm is then added
//   over its slots in slot order.  No atomics on data.
#include "common.hpp"

#include <type_traits>

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr i64 kMaxT = 4096;
constexpr uint64_t kNoKey = ~0ull;

// Exclusive scan of one int per thread over the block; returns the total.
__device__ int block_exclusive_scan(int v, int *buf, int &total)
{
    const int tid = threadIdx.x;
    buf[tid] = v;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
        const int x = tid >= off ? buf[tid - off] : 0;
        __syncthreads();
        buf[tid] += x;
        __syncthreads();
    }
    total = buf[kThreads - 1];
    const int incl = buf[tid];
    __syncthreads();
    return incl - v;
}

struct EmbWs {
    int32_t *perm;      // [N][T]   positions in sorted order
    int32_t *segstart;  // [N][T+1] first sorted index of each segment, then the end
    int32_t *segid;     // [N][T]   id of each segment
    int32_t *counts;    // [N]      distinct valid ids
    float *sqpart;      // [N][T]   squared norm of each segment slot (0 past the last)
};

__global__ __launch_bounds__(kThreads) void emb_sort_kernel(const int64_t *__restrict__ ids, i64 T,
                                                            i64 V, int P2, EmbWs w,
                                                            int32_t *status)
{
    extern __shared__ uint64_t keys[];
    __shared__ int scan_buf[kThreads];
    const i64 n = blockIdx.x;
    const int tid = threadIdx.x;
    const int64_t *idn = ids + n * T;
    bool bad = false;
    for (int i = tid; i < P2; i += kThreads) {
        uint64_t k = kNoKey;
        if (i < T) {
            const int64_t id = idn[i];
            if (id >= 0 && id < V) k = ((uint64_t)id << 32) | (uint32_t)i;
            else bad = true;
        }
        keys[i] = k;
    }
    if (bad) raise_flag(status, DP_FLAG_BAD_INDEX);
    __syncthreads();
    for (int k = 2; k <= P2; k <<= 1) {
        for (int j = k >> 1; j > 0; j >>= 1) {
            for (int i = tid; i < P2; i += kThreads) {
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
            __syncthreads();
        }
    }
    // each thread owns a contiguous range of sorted positions
    const int per = (int)((T + kThreads - 1) / kThreads);
    const int r0 = tid * per;
    const int r1 = (int)(r0 + per < T ? r0 + per : T);
    int heads = 0, valid = 0;
    for (int r = r0; r < r1; ++r) {
        const uint64_t k = keys[r];
        if (k == kNoKey) continue;
        ++valid;
        if (r == 0 || (keys[r - 1] >> 32) != (k >> 32)) ++heads;
    }
    int nseg, nvalid;
    int s = block_exclusive_scan(heads, scan_buf, nseg);
    int vtot;
    (void)block_exclusive_scan(valid, scan_buf, vtot);
    nvalid = vtot;
    int32_t *perm = w.perm + n * T;
    int32_t *seg = w.segstart + n * (T + 1);
    for (int r = r0; r < r1; ++r) {
        const uint64_t k = keys[r];
        if (k == kNoKey) continue;
        perm[r] = (int32_t)(k & 0xffffffffu);
        if (r == 0 || (keys[r - 1] >> 32) != (k >> 32)) {
            w.segid[n * T + s] = (int32_t)(k >> 32);
            seg[s++] = r;
        }
    }
    if (tid == 0) {
        seg[nseg] = nvalid;
        w.counts[n] = nseg;
    }
}

__global__ __launch_bounds__(kThreads) void emb_scan_kernel(const int32_t *__restrict__ counts,
                                                            i64 N, int64_t *__restrict__ row_ptr)
{
    __shared__ int64_t buf[kThreads];
    __shared__ int64_t carry;
    const int tid = threadIdx.x;
    if (tid == 0) {
        carry = 0;
        row_ptr[0] = 0;
    }
    __syncthreads();
    for (i64 c = 0; c < N; c += kThreads) {
        const i64 n = c + tid;
        const int64_t v = n < N ? counts[n] : 0;
        buf[tid] = v;
        __syncthreads();
        for (int off = 1; off < kThreads; off <<= 1) {
            const int64_t x = tid >= off ? buf[tid - off] : 0;
            __syncthreads();
            buf[tid] += x;
            __syncthreads();
        }
        if (n < N) row_ptr[n + 1] = carry + buf[tid];
        __syncthreads();
        if (tid == 0) carry += buf[kThreads - 1];
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

constexpr int kBatch = 8;       // positions whose loads are in flight together
constexpr int kDeepBatch = 32;  // ... for segments longer than kBatch (hot ids)

// acc += the rows perm[r0 .. r1-1] of Bn at column cc, in ascending r,
// BATCH rows' loads in flight at a time
template <typename T, int VEC, int BATCH>
__device__ __forceinline__ void sum_rows(const T *Bn, const int32_t *perm, int r0, int r1, i64 D, i64 cc,
                                         float (&acc)[VEC])
{
    for (int r = r0; r < r1; r += BATCH) {
        float v[BATCH][VEC];
#pragma unroll
        for (int j = 0; j < BATCH; ++j) {
            const int rj = r + j < r1 ? r + j : r1 - 1;
            load_vec<T, VEC>(Bn + (i64)perm[rj] * D + cc, v[j]);
        }
#pragma unroll
        for (int j = 0; j < BATCH; ++j)
            if (r + j < r1)
#pragma unroll
                for (int i = 0; i < VEC; ++i) acc[i] += v[j][i];
    }
}

template <typename T, int VEC>
__global__ __launch_bounds__(64) void emb_rows_kernel(
    const T *__restrict__ B, i64 Tn, i64 D, float scale, EmbWs w, const int64_t *__restrict__ row_ptr,
    int64_t *__restrict__ uniq, float *__restrict__ rows, i64 cap, int32_t *status)
{
    const i64 n = blockIdx.x / Tn;
    const int s = (int)(blockIdx.x % Tn);
    const int lane = threadIdx.x;
    const int u = w.counts[n];
    if (s >= u) {
        if (lane == 0) w.sqpart[n * Tn + s] = 0.0f;
        return;
    }
    const i64 k = row_ptr[n] + s;                 // CSR row of this segment
    if (s == u - 1 && k >= cap && lane == 0) raise_flag(status, DP_FLAG_CAP);
    const bool keep = k < cap;
    const int32_t *perm = w.perm + n * Tn;
    const int32_t *seg = w.segstart + n * (Tn + 1);
    const int r0 = seg[s], r1 = seg[s + 1];
    if (keep && lane == 0) uniq[k] = w.segid[n * Tn + s];

    const T *Bn = B + n * Tn * D;
    float sq = 0.0f;
    for (i64 c0 = 0; c0 < D; c0 += 64 * VEC) {
        const i64 c = c0 + (i64)VEC * lane;
        const bool on = c < D;
        const i64 cc = on ? c : 0;
        float acc[VEC];
#pragma unroll
        for (int i = 0; i < VEC; ++i) acc[i] = 0.0f;
        if (r1 - r0 > kBatch) sum_rows<T, VEC, kDeepBatch>(Bn, perm, r0, r1, D, cc, acc);
        else sum_rows<T, VEC, kBatch>(Bn, perm, r0, r1, D, cc, acc);
        if (on) {
            float g[VEC];
#pragma unroll
            for (int i = 0; i < VEC; ++i) {
                g[i] = scale * acc[i];
                sq += g[i] * g[i];
            }
            if (keep) {
                if constexpr (VEC == 4)
                    *reinterpret_cast<float4 *>(rows + k * D + c) = make_float4(g[0], g[1], g[2], g[3]);
                else
                    rows[k * D + c] = g[0];
            }
        }
    }
    sq = wave_sum(sq);
    if (lane == 0) w.sqpart[n * Tn + s] = sq;
}

EmbWs carve(void *ws, i64 N, i64 T)
{
    EmbWs w;
    char *p = (char *)ws;
    w.perm = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N * T, 256);
    w.segstart = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N * (T + 1), 256);
    w.segid = (int32_t *)p;
    p += align_up(sizeof(int32_t) * N * T, 256);
    w.counts = (int32_t *)p;
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
    return 2 * align_up(sizeof(int32_t) * N * T, 256) + align_up(sizeof(int32_t) * N * (T + 1), 256) +
           align_up(sizeof(int32_t) * N, 256) + align_up(sizeof(float) * N * T, 256);
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
    // one 64-lane workgroup per position: the grid's 2^32 work-items cap N*T
    DPG_REQUIRE(N * T < (i64(1) << 26), DP_EUNSUPPORTED);
    DPG_REQUIRE(row_ptr != nullptr, DP_EINVAL);
    DPG_REQUIRE(N * T == 0 || (ids != nullptr && B != nullptr), DP_EINVAL);
    DPG_REQUIRE(cap == 0 || (uniq_ids != nullptr && rows != nullptr), DP_EINVAL);
    const size_t need = dp_grad_sample_embedding_workspace_bytes(N, T);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0) {
        // row_ptr[0] = 0 for an empty batch
        emb_scan_kernel<<<1, kThreads, 0, stream>>>(nullptr, 0, row_ptr);
        return launch_status();
    }
    EmbWs w = carve(ws, N, T);
    int P2 = 1;
    while (P2 < T) P2 <<= 1;
    emb_sort_kernel<<<(unsigned)N, kThreads, sizeof(uint64_t) * P2, stream>>>(ids, T, V, P2, w, status);
    emb_scan_kernel<<<1, kThreads, 0, stream>>>(w.counts, N, row_ptr);
    if (T > 0) {
        const unsigned grid = (unsigned)(N * T);
        // four columns per lane when every row starts on a 16-byte (fp32) or
        // 8-byte (bf16) boundary, and rows likewise
        const bool vec = D % 4 == 0 && aligned(rows, 16) && aligned(B, dt == DP_F32 ? 16 : 8);
        if (dt == DP_F32) {
            if (vec)
                emb_rows_kernel<float, 4><<<grid, 64, 0, stream>>>((const float *)B, T, D, scale, w, row_ptr,
                                                                   uniq_ids, rows, cap, status);
            else
                emb_rows_kernel<float, 1><<<grid, 64, 0, stream>>>((const float *)B, T, D, scale, w, row_ptr,
                                                                   uniq_ids, rows, cap, status);
        } else {
            if (vec)
                emb_rows_kernel<uint16_t, 4><<<grid, 64, 0, stream>>>((const uint16_t *)B, T, D, scale, w,
                                                                      row_ptr, uniq_ids, rows, cap, status);
            else
                emb_rows_kernel<uint16_t, 1><<<grid, 64, 0, stream>>>((const uint16_t *)B, T, D, scale, w,
                                                                      row_ptr, uniq_ids, rows, cap, status);
        }
    }
    if (sqnorm) {
        if (T > 0) sum_partials(w.sqpart, N, (int)T, sqnorm, stream);
        else zero_fill(sqnorm, N, stream);
    }
    return launch_status();
}
