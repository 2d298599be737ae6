// Backward through time of an LSTM layer: the gate backprop that the per-
// sample gradients of its two weight matrices take as B.
//
// The paper's recurrent modules (DPLSTM) are its costliest per-sample layers:
// an LSTM's weights act as one Linear layer on the input x_t and one on the
// previous hidden state h_{t-1}, both fed the gradient with respect to the gate
// pre-activations z_t, and that gradient comes from the recurrence run
// backwards.  With PyTorch's gate order (i, f, g, o), zero initial state and
// the loss gradient arriving at the hidden states (dh_out at every step
// and/or dh_last at the last), for t = T-1 down to 0:
//   dh      = dh_out_t (+ dh_last at T-1) + W_hh^T delta_{t+1}   (no term at T-1)
//   dc_t    = dh * o * (1 - tanh(c_t)^2) + dc_{t+1} * f_{t+1}
//   delta_i = dc_t * g * i (1 - i)          delta_f = dc_t * c_{t-1} * f (1 - f)
//   delta_g = dc_t * i * (1 - g^2)          delta_o = dh * tanh(c_t) * o (1 - o)
//
// The steps of one sample are a chain, so the kernel is built for the
// latency of one step.  One workgroup per sample; hidden unit u is owned by
// four lanes (q = 0..3) that hold, in registers, the column W_hh[g][u] for
// their gate rows g = 4q + 16m + r (r < 4): W_hh is read once per workgroup.
// A step reads delta_{t+1} from LDS in 16-byte pieces (the four lanes of a
// unit read four different pieces, the units of a wave the same ones:
// broadcasts), multiplies it into the lane's rows in two fma chains, adds the
// four lanes' partial sums with two quad permutes, and every lane of the unit
// then runs the elementwise update (branch-free: lane q selects its gate's
// factors) and writes gate q's delta to LDS and to memory.  The step is bound
// by VALU issue (about 140 instructions per wave, two waves on three of the
// four SIMDs) and the per-step barrier and LDS latencies.  delta
// is double-buffered in LDS, so one barrier per step.  The gate activations
// and cell states of a step are loaded kRing steps ahead into a register
// ring, so their latency is hidden behind the chain.
#include "common.hpp"

namespace dpg {
namespace {

// tanh(x) = 1 - 2 / (1 + e^{2x}), from the hardware base-2 exponential and
// reciprocal (about 1e-7 absolute error; e^{2x} overflowing to infinity gives
// 1, underflowing to 0 gives -1)
__device__ __forceinline__ float tanh_exp(float x)
{
    const float e = __builtin_amdgcn_exp2f(x * 2.8853900817779268f);   // 2 log2(e)
    return 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + e);
}

constexpr int kQ = 4;          // lanes per hidden unit
constexpr int kMaxH = 128;     // 4 * 128 = 512 threads, two waves per SIMD
// MB: blocks of 16 gate rows (4H <= 16 * MB); DHO: a loss gradient at every
// hidden state is given; kRing: steps loaded ahead
template <int MB, bool DHO, int kRing = (MB > 16 ? 4 : 6)>
__global__ __launch_bounds__(512) void lstm_bptt_kernel(const float *__restrict__ gates, const float *__restrict__ c,
                                                         const float *__restrict__ W_hh,
                                                         const float *__restrict__ dh_out,
                                                         const float *__restrict__ dh_last, i64 T, int H,
                                                         float *__restrict__ delta)
{
    __shared__ __attribute__((aligned(16))) float dbuf[2][16 * MB];
    const i64 n = blockIdx.x;
    const int tid = threadIdx.x;
    const int u = tid / kQ, q = tid % kQ;
    const int G = 4 * H;
    const bool live = u < H;

    // the lane's column slice of W_hh (zero past the layer)
    float w[MB][4];
#pragma unroll
    for (int m = 0; m < MB; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int g = 4 * q + 16 * m + r;
            w[m][r] = (live && g < G) ? W_hh[(i64)g * H + u] : 0.0f;
        }
    // rows past 4H stay zero in both buffers
    for (int e = tid; e < 2 * 16 * MB; e += blockDim.x) (&dbuf[0][0])[e] = 0.0f;

    const float *gn = gates + n * T * G;
    const float *cn = c + n * T * H;
    const float *hn = DHO ? dh_out + n * T * H : nullptr;
    float *dn = delta + n * T * G;
    const float dlast = (live && dh_last) ? dh_last[n * H + u] : 0.0f;
    const int uu = live ? u : 0;               // lanes past the layer read unit 0's values

    // ring[k] = {i, f, g, o, c_t(, dh_out_t)} of a step, by raw-buffer loads
    // over the sample's arrays (32-bit offsets; a step before 0 reads zeros)
    constexpr int NV = DHO ? 6 : 5;
    float ring[kRing][NV];
    const __amdgpu_buffer_rsrc_t rg = sample_rsrc(gn, (uint32_t)(T * G) * 4u);
    const __amdgpu_buffer_rsrc_t rc = sample_rsrc(cn, (uint32_t)(T * H) * 4u);
    const __amdgpu_buffer_rsrc_t rh = sample_rsrc(DHO ? hn : cn, (uint32_t)(T * H) * 4u);
    const int hb = 4 * H;           // bytes between gate blocks
    auto load_step = [&](i64 t, float (&v)[NV]) {
        const uint32_t og = t < 0 ? kOutside : (uint32_t)(t * G + uu) * 4u;
        const uint32_t oc = t < 0 ? kOutside : (uint32_t)(t * H + uu) * 4u;
        v[0] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, og, 0, 0));
        v[1] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, og, hb, 0));
        v[2] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, og, 2 * hb, 0));
        v[3] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rg, og, 3 * hb, 0));
        v[4] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rc, oc, 0, 0));
        if constexpr (DHO) v[NV - 1] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rh, oc, 0, 0));
    };
    float dc_next = 0.0f, f_next = 0.0f;
    int cur = 0;
    // one step: dh from delta_{t+1} (the zeroed buffer at t = T-1), the
    // update, delta_t to LDS and memory
    auto step = [&](i64 t, const float (&v)[NV], float cp) {
        const float *d = dbuf[cur ^ 1];
        // the reads in three groups, each group's reads issued together
        // (measured at 4H = 400: two groups or one are slower, as are more than five)
        constexpr int HALF = (MB + 2) / 3;
        // two fma chains (even and odd rows of each 16-byte piece), added at the end
        float p0 = 0.0f, p1 = 0.0f;
#pragma unroll
        for (int m0 = 0; m0 < MB; m0 += HALF) {
            float4 x[HALF];
#pragma unroll
            for (int m = 0; m < HALF; ++m)
                if (m0 + m < MB) x[m] = *reinterpret_cast<const float4 *>(d + 4 * q + 16 * (m0 + m));
#pragma unroll
            for (int m = 0; m < HALF; ++m)
                if (m0 + m < MB) {
                    p0 = __builtin_fmaf(w[m0 + m][0], x[m].x, p0);
                    p1 = __builtin_fmaf(w[m0 + m][1], x[m].y, p1);
                    p0 = __builtin_fmaf(w[m0 + m][2], x[m].z, p0);
                    p1 = __builtin_fmaf(w[m0 + m][3], x[m].w, p1);
                }
        }
        float part = p0 + p1;
        // the unit's four lanes are a quad: two quad permutes add them
        part += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(part), 0xB1, 0xF, 0xF, false));
        part += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(part), 0x4E, 0xF, 0xF, false));
        const float gi = v[0], gf = v[1], gg = v[2], go = v[3], ct = v[4];
        const float dh = part + (DHO ? v[NV - 1] : 0.0f) + (t == T - 1 ? dlast : 0.0f);
        const float tc = tanh_exp(ct);
        const float dc = dh * go * (1.0f - tc * tc) + dc_next * f_next;
        // lane q's gate: delta_q = s1 * s2 * s3 (selects, no branches)
        const float s1 = q == 3 ? dh : dc;
        const float s2 = q == 0 ? gg : q == 1 ? cp : q == 2 ? gi : tc;
        const float gq = q == 0 ? gi : q == 1 ? gf : go;
        const float s3 = q == 2 ? 1.0f - gg * gg : gq * (1.0f - gq);
        const float val = s1 * s2 * s3;
        if (live) {
            dbuf[cur][q * H + u] = val;
            dn[t * G + q * H + u] = val;
        }
        dc_next = dc;
        f_next = gf;
        lds_barrier();
        cur ^= 1;
    };

    // full chunks of kRing steps from the end, each step's inputs loaded
    // kRing steps ahead; the weights have landed before the loop starts
#pragma unroll
    for (int k = 0; k < kRing; ++k) load_step(T - 1 - k, ring[k]);
    __builtin_amdgcn_s_waitcnt(0);
    lds_barrier();
    const i64 full = T / kRing * kRing;        // steps T-1 .. T-full
    for (i64 t0 = T - 1; t0 > T - 1 - full; t0 -= kRing) {
#pragma unroll
        for (int k = 0; k < kRing; ++k) {
            const i64 t = t0 - k;
            const float cp = t > 0 ? ring[(k + 1) % kRing][4] : 0.0f;
            step(t, ring[k], cp);
            load_step(t - kRing, ring[k]);
        }
    }
    // the remaining T mod kRing steps, loaded one at a time
    for (i64 t = T - 1 - full; t >= 0; --t) {
        float v[NV], pv[NV];
        load_step(t, v);
        load_step(t - 1, pv);
        step(t, v, t > 0 ? pv[4] : 0.0f);
    }
}

template <int MB>
void launch(const float *gates, const float *c, const float *W_hh, const float *dh_out, const float *dh_last, i64 N,
            i64 T, int H, float *delta, hipStream_t stream)
{
    const int threads = (int)ceil_div((i64)kQ * H, kWave) * kWave;
    if (dh_out)
        lstm_bptt_kernel<MB, true><<<(unsigned)N, threads, 0, stream>>>(gates, c, W_hh, dh_out, dh_last, T, H, delta);
    else
        lstm_bptt_kernel<MB, false><<<(unsigned)N, threads, 0, stream>>>(gates, c, W_hh, dh_out, dh_last, T, H,
                                                                         delta);
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" dp_status dp_lstm_backward(const float *gates, const float *c, const float *W_hh, const float *dh_out,
                                      const float *dh_last, int64_t N, int64_t T, int64_t H, float *delta,
                                      int32_t *status, hipStream_t stream)
{
    (void)status;
    DPG_REQUIRE(N >= 0 && T >= 0 && H >= 1, DP_EINVAL);
    DPG_REQUIRE(H <= kMaxH, DP_EUNSUPPORTED);
    DPG_REQUIRE(N < (i64(1) << 31) && T < (i64(1) << 40), DP_EINVAL);
    DPG_REQUIRE(T * 4 * H * 4 < (i64(1) << 31), DP_EUNSUPPORTED);   // 32-bit offsets within a sample
    DPG_REQUIRE(N * T == 0 || (gates != nullptr && c != nullptr && W_hh != nullptr && delta != nullptr),
                DP_EINVAL);
    DPG_REQUIRE(aligned(gates, 4) && aligned(c, 4) && aligned(delta, 4), DP_EINVAL);
    if (N == 0 || T == 0) return DP_OK;
    const int mb = (int)ceil_div(4 * H, 16);
    const int h = (int)H;
    if (mb <= 8)
        launch<8>(gates, c, W_hh, dh_out, dh_last, N, T, h, delta, stream);
    else if (mb <= 16)
        launch<16>(gates, c, W_hh, dh_out, dh_last, N, T, h, delta, stream);
    else if (mb <= 25)
        launch<25>(gates, c, W_hh, dh_out, dh_last, N, T, h, delta, stream);
    else
        launch<32>(gates, c, W_hh, dh_out, dh_last, N, T, h, delta, stream);
    return launch_status();
}
