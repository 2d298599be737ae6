// dp_grad_sample_linear without a caller workspace, for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation).
//
// The per-sample-gradient kernels of a Linear layer over a sequence write
// each sample's squared-norm partials (one per tile and wave) to scratch
// memory before a second kernel adds them in a fixed order.  Here that
// scratch is a file-scope device array of fixed size: every GPU the library
// runs on holds its own copy until the process ends, and its device address
// is looked up once per device with hipGetSymbolAddress (the array's name in
// host code is only a host-side stand-in).  Nothing here allocates or frees.
#include <mutex>

#include "common.hpp"

namespace dpg {

dp_status check_linear(const void *A, const void *B, dp_dtype dt, i64 N, i64 T, i64 din, i64 dout);

namespace {

constexpr size_t kScratchBytes = size_t(8) << 20;    // 8 MiB per device
constexpr int kMaxDevices = 64;

__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// The device address of this library's scratch array on the device that owns
// `stream` (the current device for the null stream), looked up on the first
// call for that device with the device current.
dp_status scratch_for(hipStream_t stream, void **out)
{
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return DP_EHIP;
    int dev = cur;
    if (stream != nullptr && hipStreamGetDevice(stream, &dev) != hipSuccess) return DP_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return DP_EUNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        if (dev != cur && hipSetDevice(dev) != hipSuccess) return DP_EHIP;
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (dev != cur && hipSetDevice(cur) != hipSuccess) return DP_EHIP;
        if (e != hipSuccess || p == nullptr) return DP_EHIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return DP_OK;
}

}  // namespace
}  // namespace dpg

using namespace dpg;

extern "C" size_t dp_grad_sample_linear_noalloc_max_bytes(void) { return kScratchBytes; }

extern "C" dp_status dp_grad_sample_linear_noalloc(const void *A, const void *B, dp_dtype dt, int64_t N,
                                                   int64_t T, int64_t d_in, int64_t d_out, float scale,
                                                   float *gW, float *gb, float *sqnorm, int32_t *status,
                                                   hipStream_t stream)
{
    dp_status st = check_linear(A, B, dt, N, T, d_in, d_out);
    if (st != DP_OK) return st;
    DPG_REQUIRE(N == 0 || gW != nullptr, DP_EINVAL);
    const size_t need = dp_grad_sample_linear_workspace_bytes(N, T, d_in, d_out, dt);
    DPG_REQUIRE(need <= kScratchBytes, DP_ECAP);
    if (need == 0 || N == 0) return dp_grad_sample_linear(A, B, dt, N, T, d_in, d_out, scale, gW, gb, sqnorm,
                                                          status, nullptr, 0, stream);
    void *ws = nullptr;
    st = scratch_for(stream, &ws);
    if (st != DP_OK) return st;
    return dp_grad_sample_linear(A, B, dt, N, T, d_in, d_out, scale, gW, gb, sqnorm, status, ws, kScratchBytes,
                                 stream);
}
