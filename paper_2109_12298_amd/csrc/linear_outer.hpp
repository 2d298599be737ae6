// Linear layer with one position per sample (T = 1): the per-sample gradient
// is the rank-one outer product
//   gW[n][i][j] = s * B[n][i] * A[n][j],   gb[n][i] = s * B[n][i],
// pure HBM write traffic (about one flop per 4 bytes written), done by a
// store-streaming workgroup body shared by the single-layer kernel and the
// grouped per-sample-gradient kernel.  The squared norm is the closed form of
// the rank-one gradient, s^2 |B_n|^2 (|A_n|^2 + 1) (the 1 only with a bias).
#pragma once

#include "common.hpp"

namespace dpg {
namespace louter {

constexpr int kThreads = 256;
constexpr int kOuterMaxRows = 1024;   // gW rows per outer-product workgroup

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

// Rows [rb * rows, rb * rows + rows) of sample n's gW (and those entries of
// gb); block rb == 0 also writes sqnorm[n] when sqnorm is not null.  VEC:
// d_in % 4 == 0 with 16-byte-aligned rows (float4 loads of A, float4 stores).
template <typename T, bool VEC>
__device__ __forceinline__ void outer_block(const T *__restrict__ A, const T *__restrict__ B, i64 din, i64 dout,
                                            int rows, i64 n, int rb, float scale, float *__restrict__ gW,
                                            float *__restrict__ gb, float *__restrict__ sqnorm)
{
    __shared__ float red[16];
    const i64 i0 = (i64)rb * rows;
    const i64 i1 = i0 + rows < dout ? i0 + rows : dout;
    __shared__ float bsh[kOuterMaxRows];
    const T *An = A + n * din;
    const T *Bn = B + n * dout;
    float *G = gW + n * dout * din;
    const bool do_norm = sqnorm != nullptr && rb == 0;

    // Every load of the block is issued before the one barrier: the sample's
    // activation (kept in registers when it fits), the block's backprop rows
    // (into LDS), and, for the norm, the whole backprop row.
    constexpr int KA = 4;
    const i64 nv = VEC ? din / 4 : 0;
    const bool inreg = VEC && nv <= (i64)kThreads * KA;
    float4 a[KA];
    float na = 0.0f, nb = 0.0f;
    if (inreg) {
#pragma unroll
        for (int k = 0; k < KA; ++k) {
            const i64 j4 = threadIdx.x + (i64)k * kThreads;
            a[k] = j4 < nv ? load4<T>(An, 4 * j4) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    if (do_norm) {
        for (i64 i = threadIdx.x; i < dout; i += kThreads) {
            const float b = load_elem<T>(Bn, i);
            nb += b * b;
        }
    }
    for (i64 i = i0 + threadIdx.x; i < i1; i += kThreads) bsh[i - i0] = scale * load_elem<T>(Bn, i);
    __syncthreads();

    if (inreg) {
#pragma unroll
        for (int k = 0; k < KA; ++k) {
            const i64 j4 = threadIdx.x + (i64)k * kThreads;
            if (j4 >= nv) break;
            na += a[k].x * a[k].x + a[k].y * a[k].y + a[k].z * a[k].z + a[k].w * a[k].w;
            for (i64 i = i0; i < i1; ++i) {
                const float b = bsh[i - i0];
                store_stream4(G + i * din + 4 * j4, b * a[k].x, b * a[k].y, b * a[k].z, b * a[k].w);
            }
        }
    } else if (VEC) {
        for (i64 j4 = threadIdx.x; j4 < nv; j4 += kThreads) {
            const float4 av = load4<T>(An, 4 * j4);
            na += av.x * av.x + av.y * av.y + av.z * av.z + av.w * av.w;
            for (i64 i = i0; i < i1; ++i) {
                const float b = bsh[i - i0];
                store_stream4(G + i * din + 4 * j4, b * av.x, b * av.y, b * av.z, b * av.w);
            }
        }
    } else {
        for (i64 j = threadIdx.x; j < din; j += kThreads) {
            const float av = load_elem<T>(An, j);
            na += av * av;
            for (i64 i = i0; i < i1; ++i) G[i * din + j] = bsh[i - i0] * av;
        }
    }
    if (gb) {
        for (i64 i = i0 + threadIdx.x; i < i1; i += kThreads) gb[n * dout + i] = bsh[i - i0];
    }
    if (do_norm) {
        // closed form of the rank-one gradient: s^2 |B_n|^2 (|A_n|^2 + 1)
        na = block_sum(na, red);
        nb = block_sum(nb, red);
        if (threadIdx.x == 0) sqnorm[n] = scale * scale * nb * (na + (gb ? 1.0f : 0.0f));
    }
}


// gW rows per workgroup and workgroups per sample for a d_in x d_out layer
struct OuterPlan {
    int rows, bps;
};

inline OuterPlan outer_plan(i64 din, i64 dout)
{
    int rows = (int)(8192 / din);
    if (rows < 1) rows = 1;
    if (rows > kOuterMaxRows) rows = kOuterMaxRows;
    if (rows > dout) rows = (int)dout;
    return OuterPlan{rows, (int)((dout + rows - 1) / rows)};
}

}  // namespace louter
}  // namespace dpg
