// Grouped per-sample gradients: the Linear (T = 1) and small Conv2d layers of
// a network in one launch.
//
// Each layer's per-sample gradient is the one of its single-layer kernel
// (the rank-one outer product of linear_outer.hpp, the one-workgroup-per-
// sample convolution of conv2d_small_dev.hpp): the same workgroup bodies, run
// by one kernel whose blocks are the concatenation of every layer's blocks.
// For small networks (the MNIST CNN: four layers, a few microseconds of work
// each) a launch's fixed costs (dispatch, the first load round trip, the
// drain) dominate; here they are paid once and the layers' workgroups overlap
// on the CUs.  Convolution layers' blocks come first, since theirs are the
// longest chains.
#include "common.hpp"
#include "conv2d_small.hpp"
#include "conv2d_small_dev.hpp"
#include "grad_sample_bf16.hpp"
#include "linear_outer.hpp"
#include "linear_staged.hpp"

namespace dpg {
namespace {

constexpr int kThreads = 256;
constexpr int kManyMax = 8;          // layers per launch (more run as further launches)
static_assert(csmall::kThreads == kThreads && louter::kThreads == kThreads, "one workgroup size");

enum { kConvSmall = 0, kOuter = 1 };

struct ManyItem {
    int kind;
    int bpw;                         // conv: accumulator blocks per wave
    int vec;                         // outer: float4 path
    int rows, bps;                   // outer: gW rows per block, blocks per sample
    i64 din, dout;                   // outer
    const void *A, *B;
    float scale;
    float *gW, *gb, *sqnorm;
    csmall::SmallShape cs;
};

struct ManyDesc {
    int count;
    int blk0[kManyMax + 1];          // first block of each layer in the launch (one scalar load)
    ManyItem it[kManyMax];
};

template <typename T>
__global__ __launch_bounds__(kThreads) void grad_many_kernel(const ManyDesc d)
{
    extern __shared__ __attribute__((aligned(16))) float lds[];
    const int b = (int)blockIdx.x;
    int p = 0;
    while (p + 1 < d.count && d.blk0[p + 1] <= b) ++p;
    const ManyItem &it = d.it[p];
    const int local = b - d.blk0[p];
    const T *A = (const T *)it.A;
    const T *B = (const T *)it.B;
    if (it.kind == kConvSmall) {
        switch (it.bpw) {
        case 1: csmall::conv_small_sample<T, 1>(A, B, it.cs, it.scale, it.gW, it.gb, it.sqnorm, local, lds); break;
        case 2: csmall::conv_small_sample<T, 2>(A, B, it.cs, it.scale, it.gW, it.gb, it.sqnorm, local, lds); break;
        case 4: csmall::conv_small_sample<T, 4>(A, B, it.cs, it.scale, it.gW, it.gb, it.sqnorm, local, lds); break;
        default: csmall::conv_small_sample<T, 8>(A, B, it.cs, it.scale, it.gW, it.gb, it.sqnorm, local, lds); break;
        }
    } else {
        const i64 n = local / it.bps;
        const int rb = local % it.bps;
        if (it.vec)
            louter::outer_block<T, true>(A, B, it.din, it.dout, it.rows, n, rb, it.scale, it.gW, it.gb, it.sqnorm);
        else
            louter::outer_block<T, false>(A, B, it.din, it.dout, it.rows, n, rb, it.scale, it.gW, it.gb, it.sqnorm);
    }
}

ConvSmallArgs conv_args(const dp_layer_grad &L, i64 N)
{
    return ConvSmallArgs{L.A, L.B, N, L.Cin, L.H, L.W, L.Cout, L.Ho, L.Wo, L.kh, L.kw, L.sh, L.sw, L.ph, L.pw};
}

// the checks of the single-layer entry points, so that nothing is enqueued
// unless every layer is valid
dp_status validate(const dp_layer_grad &L, dp_dtype dt, i64 N)
{
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    DPG_REQUIRE(N >= 0 && N < (i64(1) << 40), DP_EINVAL);
    if (L.kind == DP_LAYER_LINEAR) {
        DPG_REQUIRE(L.T >= 0 && L.T < (i64(1) << 40) && L.d_in >= 1 && L.d_out >= 1, DP_EINVAL);
        DPG_REQUIRE(N * L.T == 0 || (L.A != nullptr && L.B != nullptr), DP_EINVAL);
        DPG_REQUIRE(N == 0 || L.gW != nullptr, DP_EINVAL);
        return DP_OK;
    }
    DPG_REQUIRE(L.kind == DP_LAYER_CONV2D, DP_EINVAL);
    DPG_REQUIRE(L.Cin >= 1 && L.H >= 1 && L.W >= 1 && L.Cout >= 1, DP_EINVAL);
    DPG_REQUIRE(L.kh >= 1 && L.kw >= 1 && L.sh >= 1 && L.sw >= 1 && L.ph >= 0 && L.pw >= 0, DP_EINVAL);
    DPG_REQUIRE(L.H + 2 * L.ph >= L.kh && L.W + 2 * L.pw >= L.kw, DP_EINVAL);
    DPG_REQUIRE(L.Ho == (L.H + 2 * L.ph - L.kh) / L.sh + 1 && L.Wo == (L.W + 2 * L.pw - L.kw) / L.sw + 1,
                DP_EINVAL);
    {
        // the single-layer call's 32-bit index limit
        const i64 lim = i64(1) << 30, Hp = L.H + 2 * L.ph, Wp = L.W + 2 * L.pw;
        DPG_REQUIRE(L.Cin * Hp * Wp < lim && L.Cout * Hp * Wp < lim && L.Cin * L.kh * L.kw < lim &&
                        (Hp + 2 * L.kh) * (Wp + 2 * L.kw) < lim,
                    DP_EUNSUPPORTED);
    }
    DPG_REQUIRE(N == 0 || (L.A != nullptr && L.B != nullptr && L.gW != nullptr), DP_EINVAL);
    return DP_OK;
}

// a bf16 Linear layer over a sequence that the staged kernel takes: these
// layers share a launch of their own (bf16_grad_sample_group)
bool staged(const dp_layer_grad &L, dp_dtype dt, i64 N)
{
    return validate(L, dt, N) == DP_OK && N > 0 && L.kind == DP_LAYER_LINEAR && dt == DP_BF16 && L.T > 1 &&
           bf16_staged_ok(L.A, L.B, L.gW, N, L.T, L.d_in, L.d_out);
}

// an fp32 Linear layer over a sequence that the staged fp32 kernel takes:
// these layers share a launch of their own (fp32_grad_sample_group)
bool staged32(const dp_layer_grad &L, dp_dtype dt, i64 N)
{
    return validate(L, dt, N) == DP_OK && N > 0 && L.kind == DP_LAYER_LINEAR && dt == DP_F32 && L.T > 1 &&
           fp32_staged_ok(L.A, L.B, L.gW, N, L.T, L.d_in, L.d_out);
}

// a layer of the small-layer launch (grad_many_kernel)
bool small(const dp_layer_grad &L, dp_dtype dt, i64 N)
{
    if (validate(L, dt, N) != DP_OK || N >= (i64(1) << 24)) return false;
    if (L.kind == DP_LAYER_LINEAR) return L.T == 1 && L.d_in * L.d_out < (i64(1) << 31);
    return conv_path() == DP_CONV_AUTO && conv_small_ok(conv_args(L, N));
}

bool grouped(const dp_layer_grad &L, dp_dtype dt, i64 N)
{
    return small(L, dt, N) || staged(L, dt, N) || staged32(L, dt, N);
}

// scratch of the staged launch: each layer's squared-norm partials
size_t staged_partials_bytes(const dp_layer_grad &L, i64 N)
{
    return L.sqnorm ? align_up((size_t)N * bf16_staged_parts(L.d_in, L.d_out) * sizeof(float), 256) : 0;
}

size_t staged32_partials_bytes(const dp_layer_grad &L, i64 N)
{
    return L.sqnorm ? align_up((size_t)N * fp32_staged_parts(L.d_in, L.d_out) * sizeof(float), 256) : 0;
}

size_t single_workspace(const dp_layer_grad &L, dp_dtype dt, i64 N)
{
    if (L.kind == DP_LAYER_LINEAR) return dp_grad_sample_linear_workspace_bytes(N, L.T, L.d_in, L.d_out, dt);
    return dp_grad_sample_conv2d_workspace_bytes(N, L.Cin, L.H, L.W, L.Cout, L.kh, L.kw, L.sh, L.sw, L.ph, L.pw);
}

void fill_item(const dp_layer_grad &L, dp_dtype dt, i64 N, ManyItem &it)
{
    it.A = L.A;
    it.B = L.B;
    it.scale = L.scale;
    it.gW = L.gW;
    it.gb = L.gb;
    it.sqnorm = L.sqnorm;
    it.bpw = 1;
    it.vec = 0;
    it.rows = it.bps = 1;
    it.din = it.dout = 0;
    it.cs = csmall::SmallShape{};
    if (L.kind == DP_LAYER_CONV2D) {
        it.kind = kConvSmall;
        csmall::make_small(conv_args(L, N), it.cs);
        it.cs.vec = it.cs.KK % 4 == 0 && aligned(L.gW, 16);
        it.cs.xdma = it.cs.xplain && dt == DP_F32 && aligned(L.A, 16);
        it.cs.gdma = it.cs.gplain && dt == DP_F32 && aligned(L.B, 16);
        it.bpw = it.cs.bpw;
    } else {
        it.kind = kOuter;
        const louter::OuterPlan op = louter::outer_plan(L.d_in, L.d_out);
        it.rows = op.rows;
        it.bps = op.bps;
        it.din = L.d_in;
        it.dout = L.d_out;
        it.vec = (L.d_in % 4) == 0 && aligned(L.A, dt == DP_F32 ? 16 : 8) && aligned(L.gW, 16);
    }
}

void launch_group(const dp_layer_grad *const *layers, int count, dp_dtype dt, i64 N, hipStream_t stream)
{
    ManyDesc d;
    d.count = count;
    i64 blocks = 0;
    size_t lds = 0;
    for (int k = 0; k < count; ++k) {
        ManyItem &it = d.it[k];
        fill_item(*layers[k], dt, N, it);
        d.blk0[k] = (int)blocks;
        blocks += it.kind == kConvSmall ? N : N * it.bps;
        if (it.kind == kConvSmall) {
            const size_t need = (size_t)csmall::lds_floats(it.cs) * sizeof(float);
            lds = need > lds ? need : lds;
        }
    }
    for (int k = count; k <= kManyMax; ++k) d.blk0[k] = (int)blocks;
    for (int k = count; k < kManyMax; ++k) d.it[k] = d.it[0];
    if (dt == DP_BF16)
        grad_many_kernel<uint16_t><<<(unsigned)blocks, kThreads, lds, stream>>>(d);
    else
        grad_many_kernel<float><<<(unsigned)blocks, kThreads, lds, stream>>>(d);
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" int32_t dp_grad_sample_many_grouped(const dp_layer_grad *item, dp_dtype dt, int64_t N)
{
    return item != nullptr && grouped(*item, dt, N) ? 1 : 0;
}

extern "C" size_t dp_grad_sample_many_workspace_bytes(const dp_layer_grad *items, int32_t count, dp_dtype dt,
                                                      int64_t N)
{
    size_t need = 0;
    if (items == nullptr || count < 0) return 0;
    // the staged layers' partials, per launch of up to kBf16GroupMax layers;
    // the single-layer calls reuse the same scratch afterwards
    size_t launch = 0;
    int in_launch = 0;
    for (int k = 0; k < count; ++k) {
        if (!staged(items[k], dt, N)) continue;
        if (in_launch == kBf16GroupMax) {
            launch = 0;
            in_launch = 0;
        }
        launch += staged_partials_bytes(items[k], N);
        ++in_launch;
        need = launch > need ? launch : need;
    }
    launch = 0;
    in_launch = 0;
    for (int k = 0; k < count; ++k) {
        if (!staged32(items[k], dt, N)) continue;
        if (in_launch == kPsGroupMax) {
            launch = 0;
            in_launch = 0;
        }
        launch += staged32_partials_bytes(items[k], N);
        ++in_launch;
        need = launch > need ? launch : need;
    }
    for (int k = 0; k < count; ++k) {
        if (grouped(items[k], dt, N) || validate(items[k], dt, N) != DP_OK) continue;
        const size_t w = single_workspace(items[k], dt, N);
        need = w > need ? w : need;
    }
    return need;
}

extern "C" dp_status dp_grad_sample_many(const dp_layer_grad *items, int32_t count, dp_dtype dt, int64_t N,
                                         int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream)
{
    DPG_REQUIRE(count >= 0 && count <= 64 && (count == 0 || items != nullptr), DP_EINVAL);
    DPG_REQUIRE(dtype_ok(dt), DP_EDTYPE);
    for (int k = 0; k < count; ++k) {
        const dp_status st = validate(items[k], dt, N);
        if (st != DP_OK) return st;
    }
    const size_t need = dp_grad_sample_many_workspace_bytes(items, count, dt, N);
    DPG_REQUIRE(ws_bytes >= need && (need == 0 || ws != nullptr), DP_EINVAL);
    if (N == 0 || count == 0) return DP_OK;

    // small layers, convolutions first, in launches of up to kManyMax
    const dp_layer_grad *order[64];
    int ng = 0;
    for (int pass = 0; pass < 2; ++pass)
        for (int k = 0; k < count; ++k)
            if (small(items[k], dt, N) && (items[k].kind == DP_LAYER_CONV2D) == (pass == 0)) order[ng++] = &items[k];
    for (int k0 = 0; k0 < ng; k0 += kManyMax)
        launch_group(order + k0, ng - k0 < kManyMax ? ng - k0 : kManyMax, dt, N, stream);
    dp_status st = launch_status();
    if (st != DP_OK) return st;

    // bf16 sequence layers, in launches of up to kBf16GroupMax, their norm
    // partials laid out one layer after another in the scratch
    {
        Bf16GroupLayer grp[kBf16GroupMax];
        int n = 0;
        size_t off = 0;
        auto flush = [&]() {
            bf16_grad_sample_group(grp, n, N, stream);
            n = 0;
            off = 0;
        };
        for (int k = 0; k < count; ++k) {
            const dp_layer_grad &L = items[k];
            if (!staged(L, dt, N)) continue;
            if (n == kBf16GroupMax) flush();
            grp[n++] = Bf16GroupLayer{L.A, L.B, L.T, L.d_in, L.d_out, L.scale, L.gW, L.gb, L.sqnorm,
                                      L.sqnorm ? (float *)((char *)ws + off) : nullptr};
            off += staged_partials_bytes(L, N);
        }
        if (n) flush();
        st = launch_status();
        if (st != DP_OK) return st;
    }

    // fp32 sequence layers on the staged kernel, in launches of up to
    // kPsGroupMax, their norm partials one layer after another in the scratch
    {
        Fp32GroupLayer grp[kPsGroupMax];
        int n = 0;
        size_t off = 0;
        auto flush = [&]() {
            fp32_grad_sample_group(grp, n, N, stream);
            n = 0;
            off = 0;
        };
        for (int k = 0; k < count; ++k) {
            const dp_layer_grad &L = items[k];
            if (!staged32(L, dt, N)) continue;
            if (n == kPsGroupMax) flush();
            grp[n++] = Fp32GroupLayer{L.A, L.B, L.T, L.d_in, L.d_out, L.scale, L.gW, L.gb, L.sqnorm,
                                      L.sqnorm ? (float *)((char *)ws + off) : nullptr};
            off += staged32_partials_bytes(L, N);
        }
        if (n) flush();
        st = launch_status();
        if (st != DP_OK) return st;
    }

    // the others through their single-layer entry points
    for (int k = 0; k < count && st == DP_OK; ++k) {
        const dp_layer_grad &L = items[k];
        if (grouped(L, dt, N)) continue;
        if (L.kind == DP_LAYER_LINEAR)
            st = dp_grad_sample_linear(L.A, L.B, dt, N, L.T, L.d_in, L.d_out, L.scale, L.gW, L.gb, L.sqnorm, status, ws,
                                       ws_bytes, stream);
        else
            st = dp_grad_sample_conv2d(L.A, L.B, dt, N, L.Cin, L.H, L.W, L.Cout, L.Ho, L.Wo, L.kh, L.kw, L.sh, L.sw,
                                       L.ph, L.pw, 1, 1, 1, L.scale, L.gW, L.gb, L.sqnorm, status, ws, ws_bytes,
                                       stream);
    }
    return st;
}
