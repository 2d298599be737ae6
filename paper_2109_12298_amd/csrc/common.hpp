// Shared device/host helpers of libdpgrad (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dpgrad.h"

namespace dpg {

typedef int64_t i64;

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// host-side argument checks (no HIP call happens before these pass)
// ---------------------------------------------------------------------------
#define DPG_REQUIRE(cond, code)                                                    \
    do {                                                                           \
        if (!(cond)) return (code);                                                \
    } while (0)

inline bool dtype_ok(dp_dtype dt) { return dt == DP_F32 || dt == DP_BF16; }
inline size_t dtype_bytes(dp_dtype dt) { return dt == DP_BF16 ? 2 : 4; }

inline dp_status launch_status()
{
    hipError_t e = hipGetLastError();
    return e == hipSuccess ? DP_OK : DP_EHIP;
}

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline bool aligned(const void *p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

__host__ __device__ inline i64 ceil_div(i64 a, i64 b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------
// element loads (bf16 is carried as its raw 16 bits)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t b)
{
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

template <typename T>
__device__ __forceinline__ float load_elem(const T *p, i64 i);

template <>
__device__ __forceinline__ float load_elem<float>(const float *p, i64 i)
{
    return p[i];
}

template <>
__device__ __forceinline__ float load_elem<uint16_t>(const uint16_t *p, i64 i)
{
    return bf16_to_f32(p[i]);
}

// A 16-byte store marked non-temporal (streamed past the caches), for large
// outputs that the next kernel reads from memory anyway.
__device__ __forceinline__ void store_stream4(float *p, float a, float b, float c, float d)
{
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    const f32x4_t v = {a, b, c, d};
    __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t *>(p));
}

// A 16-byte load marked non-temporal, for data read once.
__device__ __forceinline__ float4 load_stream4(const float *p)
{
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    const f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t *>(p));
    return make_float4(v[0], v[1], v[2], v[3]);
}

// ---------------------------------------------------------------------------
// XCD-aware block order.  Workgroups are dispatched round-robin over the 8
// XCDs (each with its own L2): block b runs on XCD b % 8.  Renumbering so that
// XCD x gets a contiguous range of logical blocks keeps neighbouring tiles,
// which share operand tiles, in one L2.  A bijection on [0, nb).
// ---------------------------------------------------------------------------
constexpr int kXcds = 8;

__device__ __forceinline__ i64 xcd_swizzle(i64 b, i64 nb)
{
    const i64 q = nb / kXcds, r = nb % kXcds;
    const i64 x = b % kXcds, k = b / kXcds;
    return x * q + (x < r ? x : r) + k;
}

// ---------------------------------------------------------------------------
// device-side status flags (rare: only on bad input)
// ---------------------------------------------------------------------------
__device__ __forceinline__ void raise_flag(int32_t *status, int32_t flag)
{
    if (status) atomicOr(status, flag);
}

// Clip factor min(1, C / (norm + 1e-6)) in fp32; C = +inf gives 1 and a
// non-finite norm gives NaN (never silently 1).
// A negative norm marks a sample outside the active batch (a padded row of
// a batch of variable size): its factor is 0, so it adds nothing.
__device__ __forceinline__ float clip_factor(float norm, float C)
{
    if (norm < 0.0f) return 0.0f;
    if (!isfinite(norm)) return __builtin_nanf("");
    if (isinf(C)) return 1.0f;
    float q = C / (norm + 1e-6f);
    return q < 1.0f ? q : 1.0f;
}

// A workgroup barrier that orders LDS only.  __syncthreads() also waits for
// every outstanding global access of the wave, loads in flight and stores
// not yet acknowledged alike; this one leaves them outstanding.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Raw-buffer descriptor over an array of `bytes` bytes (gfx9 word for 32-bit
// untyped accesses): a load at a byte offset at or past `bytes` reads zero,
// so bounded loads need no branch (and no wait at the branch's join).
// kOutside is an offset that is always past the end.
constexpr uint32_t kOutside = 0x80000000u;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t sample_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ int32_t buffer_load_i32(__amdgpu_buffer_rsrc_t r, uint32_t byte_offset)
{
    return __builtin_amdgcn_raw_buffer_load_b32(r, byte_offset, 0, 0);
}

// ---------------------------------------------------------------------------
// fixed-order reductions
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v)
{
    // butterfly over the 64 lanes; every lane ends with the same value and the
    // order of additions depends only on lane positions (deterministic)
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

// Sum over a block of `nthreads` (multiple of 64, <= 1024). Result valid in all
// threads. `red` is __shared__ float[16].
__device__ __forceinline__ float block_sum(float v, float *red)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wid = threadIdx.x / kWave;
    const int nw = (blockDim.x + kWave - 1) / kWave;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[wid] = v;
    __syncthreads();
    float s = 0.0f;
    for (int w = 0; w < nw; ++w) s += red[w];
    return s;
}

// sum_k p[k * stride] for k = 0 .. count-1, added in ascending k, with eight
// loads in flight at a time (a loop of dependent single loads is bound by
// memory latency, not bandwidth).
__device__ __forceinline__ float ordered_sum(const float *__restrict__ p, i64 stride, int count)
{
    float s = 0.0f;
    for (int k = 0; k < count; k += 8) {
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = k + j < count ? p[(i64)(k + j) * stride] : 0.0f;
#pragma unroll
        for (int j = 0; j < 8; ++j) s += v[j];
    }
    return s;
}

// One wave per sample: sqnorm[n] = sum of the sample's `parts` tile partials
// (lane l adds partials l, l+64, ... in order, then a fixed butterfly).
template <int Unused = 0>
__global__ void sum_partials_kernel(const float *__restrict__ partial, i64 N, int parts,
                                    float *__restrict__ sqnorm)
{
    const i64 n = (i64)blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave;
    const int lane = threadIdx.x & (kWave - 1);
    if (n >= N) return;
    const float *p = partial + n * parts;
    float s = 0.0f;
    for (int t = lane; t < parts; t += kWave) s += p[t];
    s = wave_sum(s);
    if (lane == 0) sqnorm[n] = s;
}

inline void sum_partials(const float *partial, i64 N, int parts, float *sqnorm, hipStream_t stream)
{
    const int per_block = 4;
    sum_partials_kernel<0><<<(unsigned)((N + per_block - 1) / per_block), per_block * kWave, 0, stream>>>(
        partial, N, parts, sqnorm);
}

// ---------------------------------------------------------------------------
// zero fill by a kernel (kept out of hipMemsetAsync so that callers may
// capture the launches in a HIP graph)
// ---------------------------------------------------------------------------
template <int Unused = 0>
__global__ void fill_zero_kernel(float *__restrict__ p, i64 n)
{
    for (i64 i = (i64)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (i64)gridDim.x * blockDim.x)
        p[i] = 0.0f;
}

inline void zero_fill(float *p, i64 n, hipStream_t stream)
{
    if (p == nullptr || n <= 0) return;
    i64 blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    fill_zero_kernel<0><<<(unsigned)blocks, 256, 0, stream>>>(p, n);
}

}  // namespace dpg
