// fp32 MFMA tile core shared by the per-sample GEMM kernels.
//
// A workgroup of 256 threads (4 waves of 64) owns a BM x BN output tile,
// split 2 x 2 over the waves; each wave covers (BM/2) x (BN/2) with 32x32
// blocks of v_mfma_f32_32x32x2_f32.  Both operand tiles are staged in LDS
// K-major ("[k][m]" and "[k][n]"), which is the order the per-sample
// contractions read them in global memory (activations and backprops are
// [positions][features]), so the MFMA operand fetch needs no transpose.
//
// Operand layout of v_mfma_f32_32x32x2_f32 (wave64): lane l supplies
// A[i = l % 32][k = l / 32] and B[k = l / 32][j = l % 32]; accumulator
// register r of lane l holds C[i][j] with j = l % 32 and
// i = 8 * (r / 4) + 4 * (l / 32) + (r % 4).
#pragma once

#include "common.hpp"

namespace dpg {

typedef float f32x16 __attribute__((ext_vector_type(16)));

template <int BM, int BN>
struct MfmaTile {
    static constexpr int WM = BM / 2;      // wave tile rows
    static constexpr int WN = BN / 2;      // wave tile cols
    static constexpr int FM = WM / 32;     // 32x32 blocks per wave, rows
    static constexpr int FN = WN / 32;     // 32x32 blocks per wave, cols
    static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32");

    f32x16 acc[FM][FN];

    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
            for (int b = 0; b < FN; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
    }

    // As: [BK][lda] (k-major over the BM rows), Bs: [BK][ldb].
    template <int BK>
    __device__ __forceinline__ void mma(const float *As, int lda, const float *Bs, int ldb,
                                        int wm, int wn, int lane)
    {
        const int li = lane & 31;
        const int lk = lane >> 5;
#pragma unroll
        for (int kk = 0; kk < BK; kk += 2) {
            float a[FM], b[FN];
#pragma unroll
            for (int x = 0; x < FM; ++x) a[x] = As[(kk + lk) * lda + wm + x * 32 + li];
#pragma unroll
            for (int y = 0; y < FN; ++y) b[y] = Bs[(kk + lk) * ldb + wn + y * 32 + li];
#pragma unroll
            for (int x = 0; x < FM; ++x)
#pragma unroll
                for (int y = 0; y < FN; ++y)
                    acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[x], b[y], acc[x][y], 0, 0, 0);
        }
    }

    // Visit every accumulator with its (row, col) inside the BM x BN tile.
    template <typename F>
    __device__ __forceinline__ void for_each(int wm, int wn, int lane, F &&f) const
    {
        const int lj = lane & 31;
        const int lh = lane >> 5;
#pragma unroll
        for (int x = 0; x < FM; ++x)
#pragma unroll
            for (int y = 0; y < FN; ++y)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = wm + x * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
                    const int col = wn + y * 32 + lj;
                    f(row, col, acc[x][y][r]);
                }
    }
};

}  // namespace dpg
