// Staging of bf16 operand tiles in LDS for the MFMA kernels that contract
// over rows of K-major ([row][feature], feature contiguous) activations and
// backprops: the fused clipped sum (clipsum_many.hip) and the per-sample
// gradients (linear_bf16.hip).
//
// Stages.  A stage is BK = 32 consecutive rows of the A tile (BMJ features)
// and of the B tile (BNI features), copied straight from global memory into
// LDS by global_load_lds_dwordx4: 16 bytes per lane, 1 KB per wave
// instruction, no VGPR round trip.  Inside a row, 16-byte chunk q is stored
// at chunk position q ^ (4 * (row & 3)).
//
// Operands.  v_mfma_f32_32x32x16_bf16 takes, per lane, eight consecutive
// rows of one feature.  gfx950's transposing LDS read ds_read_b64_tr_b16
// delivers them: within each 16-lane group, lane s reads four features of row
// s/4, and lane i receives feature i of those four rows; two reads (rows r
// and r+4) make one operand.  With the swizzle above, the four rows of a read
// put their 64-byte pieces in four different quarters of the 256-byte bank
// window, so the reads are free of bank conflicts.
//
// Accumulators: MFMA rows run over A's features (j), columns over B's (i);
// register r of lane l holds j = 8*(r/4) + 4*(l/32) + r%4, i = l%32 of its
// 32x32 block, so four consecutive registers are four consecutive j.
#pragma once

#include "common.hpp"

// the stage loads clobber M0 on purpose (see dma16)
#pragma clang diagnostic ignored "-Winline-asm"

namespace dpg {
namespace bf16s {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef short i16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;

constexpr int BK = 32;    // rows per stage (two k-steps of 16)

// byte offset of (row t, feature f) in a swizzled staged tile of row length `row_bytes`
__device__ __forceinline__ int swz(int t, int f, int row_bytes)
{
    return t * row_bytes + 16 * ((f >> 3) ^ (4 * (t & 3))) + 2 * (f & 7);
}

// One MFMA operand: rows t_base + 8 * (lane / 32) .. +7 of feature
// f_base + lane % 32, from two transposing reads of four rows each.
__device__ __forceinline__ bf16x8_t read_operand(const char *L, int row_bytes, int t_base, int f_base, int lane)
{
    const int g = lane >> 4, s = lane & 15;
    const int t = t_base + 8 * (g >> 1) + (s >> 2);
    const int f = f_base + 16 * (g & 1) + 4 * (s & 3);
    const i16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(L + swz(t, f, row_bytes)));
    const i16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t *)(L + swz(t + 4, f, row_bytes)));
    const i16x8_t v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8_t, v);
}

// A wave's operands of one k-step: FM 32-feature blocks of A, FN of B.
template <int FM, int FN>
struct Frag {
    bf16x8_t a[FM], b[FN];
};

// The operands of k-step ks (rows 16*ks .. 16*ks+15) of the stage at L (A
// tile first, B tile at byte a_bytes), for the wave's features wj.. (A) and
// wi.. (B).
template <int FM, int FN, int A_ROW, int B_ROW, int A_BYTES>
__device__ __forceinline__ void load_frag(const char *L, int ks, int wj, int wi, int lane, Frag<FM, FN> &f)
{
#pragma unroll
    for (int x = 0; x < FM; ++x) f.a[x] = read_operand(L, A_ROW, 16 * ks, wj + 32 * x, lane);
#pragma unroll
    for (int y = 0; y < FN; ++y) f.b[y] = read_operand(L + A_BYTES, B_ROW, 16 * ks, wi + 32 * y, lane);
}

template <int FM, int FN>
__device__ __forceinline__ void mma(const Frag<FM, FN> &f, f32x16_t (&acc)[FM][FN])
{
#pragma unroll
    for (int x = 0; x < FM; ++x)
#pragma unroll
        for (int y = 0; y < FN; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[x], f.b[y], acc[x][y], 0, 0, 0);
}

// Ask the scheduler to issue a k-step's 2*(FM+FN) operand reads between its
// FM*FN MFMAs (one MFMA, two reads, ...), so the reads issue while the
// matrix unit works instead of in a burst that leaves it idle.
template <int FM, int FN>
__device__ __forceinline__ void interleave_reads_with_mfma()
{
    constexpr int pairs = FM + FN;        // read pairs
    constexpr int mfma = FM * FN;
    static_assert(pairs <= mfma, "at most one read pair per MFMA");
#pragma unroll
    for (int i = 0; i < pairs; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);   // two LDS reads
    }
    __builtin_amdgcn_sched_group_barrier(0x008, mfma - pairs, 0);
}

__device__ __forceinline__ void wait_lgkmcnt0()
{
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// s_waitcnt vmcnt(n) for a run-time n in [0, 63] (the count is an
// instruction immediate: one branch per value, taken on the scalar unit)
template <int K = 0>
__device__ __forceinline__ void wait_vmcnt_rt(int n)
{
    if constexpr (K < 63) {
        if (n == K) {
            wait_vmcnt<K>();
            return;
        }
        wait_vmcnt_rt<K + 1>(n);
    } else {
        wait_vmcnt<63>();
    }
}

// Wait until a stage's loads have landed when up to four stages are staged
// (so at most two later stages have been issued): `later` stages exist after
// it, LOADS loads per stage per wave.
template <int LOADS>
__device__ __forceinline__ void wait_stages_after(int later)
{
    if (later >= 2) wait_vmcnt<2 * LOADS>();
    else if (later == 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
}

__device__ __forceinline__ void stage_barrier()
{
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// One global_load_lds_dwordx4: lane l's 16 bytes at `src` go to LDS byte
// lds + 16 * l (lds is wave-uniform and goes through M0).  Written as inline
// assembly so that the compiler, which cannot tell which LDS bytes such a
// load writes, does not wait for every outstanding stage before each LDS
// read; the stage pipelines wait for exactly the loads they need.
__device__ __forceinline__ void dma16(const void *src, uint32_t lds)
{
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src),
                 "s"(__builtin_amdgcn_readfirstlane(lds))
                 : "memory", "m0");
}

// LDS byte address (what M0 takes) of a __shared__ object
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(T *p)
{
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)p;
}

// A wave's share of the direct loads of one stage of a BMJ x BNI tile pair:
// per-lane element offsets (row-in-stage * row length + feature) and LDS
// byte offsets.  A wave-instruction covers 1 KB: 1024 / (2 BMJ) rows of A or
// 1024 / (2 BNI) rows of B; wave w takes instructions w, w + WAVES, ...
// Features past the layer's end read a clamped valid chunk (their outputs
// are never stored; d % 8 == 0 keeps chunks all-in or all-out).
template <int BMJ, int BNI, int WAVES>
struct StagePlan {
    static constexpr int A_ROW = BMJ * 2, B_ROW = BNI * 2;
    static constexpr int A_BYTES = BK * A_ROW, B_BYTES = BK * B_ROW;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int A_INSTR = A_BYTES / 1024 / WAVES, B_INSTR = B_BYTES / 1024 / WAVES;
    static constexpr int LOADS = A_INSTR + B_INSTR;
    static_assert(A_INSTR * WAVES * 1024 == A_BYTES && B_INSTR * WAVES * 1024 == B_BYTES, "stage split");
    static constexpr int A_RPI = 1024 / A_ROW, B_RPI = 1024 / B_ROW;    // rows per instruction
    static constexpr int A_CPR = A_ROW / 16, B_CPR = B_ROW / 16;        // 16-byte chunks per row

    int offA[A_INSTR], offB[B_INSTR];
    uint32_t ldsA[A_INSTR], ldsB[B_INSTR];

    __device__ __forceinline__ StagePlan(i64 din, i64 dout, i64 m0, i64 n0, int wave, int lane)
    {
#pragma unroll
        for (int r = 0; r < A_INSTR; ++r) {
            const int a = wave + WAVES * r;
            const int t = A_RPI * a + lane / A_CPR;
            const int q = (lane % A_CPR) ^ (4 * (t & 3));
            i64 f = m0 + 8 * q;
            f = f < din ? f : din - 8;
            offA[r] = (int)(t * din + f);
            ldsA[r] = (uint32_t)(a * 1024);
        }
#pragma unroll
        for (int r = 0; r < B_INSTR; ++r) {
            const int a = wave + WAVES * r;
            const int t = B_RPI * a + lane / B_CPR;
            const int q = (lane % B_CPR) ^ (4 * (t & 3));
            i64 f = n0 + 8 * q;
            f = f < dout ? f : dout - 8;
            offB[r] = (int)(t * dout + f);
            ldsB[r] = (uint32_t)(A_BYTES + a * 1024);
        }
    }

    // issue the loads of rows k0 .. k0+31 of A [.][din] and B [.][dout] into the stage at LDS byte L
    __device__ __forceinline__ void issue(const uint16_t *A, const uint16_t *B, i64 din, i64 dout, i64 k0,
                                          uint32_t L) const
    {
        const uint16_t *a = A + k0 * din;
        const uint16_t *b = B + k0 * dout;
#pragma unroll
        for (int r = 0; r < A_INSTR; ++r) dma16(a + offA[r], L + ldsA[r]);
#pragma unroll
        for (int r = 0; r < B_INSTR; ++r) dma16(b + offB[r], L + ldsB[r]);
    }
};

}  // namespace bf16s
}  // namespace dpg
