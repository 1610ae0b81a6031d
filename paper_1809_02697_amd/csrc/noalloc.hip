// The blocked convolution for callers that cannot allocate device memory:
// its split-reduction partials live in a fixed device array instead of a
// workspace the library allocates.
#include <mutex>
#include <string>

#include "neo_internal.h"

namespace {

// Partial sums of a split reduction, [split][N][KB][OH][OW][16] floats; every
// call on a device shares that device's copy.
constexpr size_t kScratchBytes = (size_t)NEO_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) float scratch[kScratchBytes / sizeof(float)];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
float* g_scratch[kMaxDevices];  // the array's device address on each device, once looked up

// The device address of the current device's copy of `scratch`.  In host code
// the array's name is only a stand-in for the symbol, so its address is taken
// from the runtime once per device, with that device current.
int scratch_of_current_device(float** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return neo::hip_fail(e, "neo_conv2d_blocked_noalloc: hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices)
        return neo::fail(NEO_ERR_UNSUPPORTED, "neo_conv2d_blocked_noalloc: device index above 63");
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return neo::hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                                 "neo_conv2d_blocked_noalloc: hipGetSymbolAddress(scratch)");
        g_scratch[dev] = static_cast<float*>(p);
    }
    *out = g_scratch[dev];
    return NEO_OK;
}

}  // namespace

extern "C" int neo_conv2d_blocked_noalloc(const float* x, int N, int C, int H, int W,
                                          const float* w_packed, int K, int R, int S,
                                          const float* bias, int stride_h, int stride_w, int pad_h,
                                          int pad_w, const neo_epilogue* ep, float* y,
                                          int y_cblk_offset, int y_cblk_total,
                                          neo_stream_t stream) {
    using namespace neo;
    ConvShape s;
    ConvConfig cfg;
    const float* res = nullptr;
    int rc = conv_prepare("neo_conv2d_blocked_noalloc", x, 16, N, C, H, W, w_packed, K, R, S, bias,
                          stride_h, stride_w, pad_h, pad_w, ep, y, 16, y_cblk_offset, y_cblk_total,
                          &s, &cfg, &res);
    if (rc != NEO_OK) return rc;
    float* ws = nullptr;
    if (cfg.split > 1) {
        const size_t need = conv_workspace_bytes(s, cfg);
        if (need > kScratchBytes)
            return fail(NEO_ERR_UNSUPPORTED,
                        "neo_conv2d_blocked_noalloc: the split reduction needs " +
                            std::to_string(need) + " bytes of partial sums, above the fixed " +
                            std::to_string(kScratchBytes) + "-byte scratch array; use "
                            "neo_conv2d_blocked");
        rc = scratch_of_current_device(&ws);
        if (rc != NEO_OK) return rc;
    }
    // Every partial element the reduce pass reads is written by exactly one
    // workgroup of this launch, so the array needs no clearing between calls.
    hipError_t e = launch_conv2d(s, cfg, x, w_packed, false, bias, res, y, ws, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_conv2d_blocked_noalloc launch");
}
