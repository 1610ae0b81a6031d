// C-ABI entry points of libneo: argument validation, then the launchers.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <limits>
#include <map>
#include <mutex>
#include <string>
#include <utility>

#include "neo_internal.h"

namespace neo {

static thread_local std::string g_err;

void set_error(const std::string& msg) { g_err = msg; }

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

int hip_fail(hipError_t e, const char* what) {
    g_err = std::string(what) + ": " + hipGetErrorString(e);
    return NEO_ERR_HIP;
}

void fold_bn_host(const float* w, const float* bias, const float* gamma, const float* beta,
                  const float* mean, const float* var, float eps, int K, int C, int R, int S,
                  float* w_out, float* bias_out) {
    const long per_k = (long)C * R * S;
    for (int k = 0; k < K; ++k) {
        const double scale = (double)gamma[k] / std::sqrt((double)var[k] + (double)eps);
        for (long i = 0; i < per_k; ++i)
            w_out[k * per_k + i] = (float)((double)w[k * per_k + i] * scale);
        const double b = bias ? (double)bias[k] : 0.0;
        bias_out[k] = (float)((b - (double)mean[k]) * scale + (double)beta[k]);
    }
}

void pack_filter_host(const float* w, int K, int C, int R, int S, int ib, int ob, float* out) {
    const int KB = cdiv(K, ob), CB = cdiv(C, ib);
    long t = 0;
    for (int kb = 0; kb < KB; ++kb)
        for (int cb = 0; cb < CB; ++cb)
            for (int r = 0; r < R; ++r)
                for (int s = 0; s < S; ++s)
                    for (int ci = 0; ci < ib; ++ci)
                        for (int ko = 0; ko < ob; ++ko, ++t) {
                            const int k = kb * ob + ko, c = cb * ib + ci;
                            out[t] = (k < K && c < C) ? w[(((long)k * C + c) * R + r) * S + s] : 0.f;
                        }
}

void blocks_to_mfma_order(const float* in, long n_blocks, float* out) {
    for (long b = 0; b < n_blocks; ++b)
        for (int c = 0; c < 16; ++c)
            for (int k = 0; k < 16; ++k)
                out[b * 256 + ((c / 4) * 16 + k) * 4 + c % 4] = in[b * 256 + c * 16 + k];
}

void blocks_from_mfma_order(const float* in, long n_blocks, float* out) {
    for (long b = 0; b < n_blocks; ++b)
        for (int c = 0; c < 16; ++c)
            for (int k = 0; k < 16; ++k)
                out[b * 256 + c * 16 + k] = in[b * 256 + ((c / 4) * 16 + k) * 4 + c % 4];
}

long kernel_filter_floats(const ConvShape& s) {
    const long KB = cdiv(s.K, 16);
    if (conv_small_c(s)) return KB * s.R * cdiv(s.S, 4) * 256;
    return KB * cdiv(s.C, 16) * s.R * s.S * 256;
}

// Small-channel order: the block of (kb, r, u) holds, for lane (k, g), the
// float4 w[k][c = 0..3][r][s = 4u + g]; the KCRS[16]c[16]k source has one
// channel block, its block (kb, r, s) at ((kb * R + r) * S + s) * 256, [c][k].
void to_kernel_order(const float* packed, const ConvShape& s, float* out) {
    if (!conv_small_c(s)) {
        blocks_to_mfma_order(packed, kernel_filter_floats(s) / 256, out);
        return;
    }
    const int KB = cdiv(s.K, 16), U = cdiv(s.S, 4);
    for (int kb = 0; kb < KB; ++kb)
        for (int r = 0; r < s.R; ++r)
            for (int u = 0; u < U; ++u)
                for (int g = 0; g < 4; ++g)
                    for (int k = 0; k < 16; ++k)
                        for (int c = 0; c < 4; ++c) {
                            const int sc = 4 * u + g;
                            const long o = (((long)(kb * s.R + r) * U + u) * 4 + g) * 64 + k * 4 + c;
                            out[o] = sc < s.S
                                         ? packed[((long)(kb * s.R + r) * s.S + sc) * 256 + c * 16 + k]
                                         : 0.f;
                        }
}

void from_kernel_order(const float* in, const ConvShape& s, float* packed) {
    if (!conv_small_c(s)) {
        blocks_from_mfma_order(in, kernel_filter_floats(s) / 256, packed);
        return;
    }
    const int KB = cdiv(s.K, 16), U = cdiv(s.S, 4);
    std::fill(packed, packed + (long)KB * s.R * s.S * 256, 0.f);  // channels 4..15 are padding
    for (int kb = 0; kb < KB; ++kb)
        for (int r = 0; r < s.R; ++r)
            for (int sc = 0; sc < s.S; ++sc)
                for (int k = 0; k < 16; ++k)
                    for (int c = 0; c < 4; ++c) {
                        const int u = sc / 4, g = sc % 4;
                        packed[((long)(kb * s.R + r) * s.S + sc) * 256 + c * 16 + k] =
                            in[(((long)(kb * s.R + r) * U + u) * 4 + g) * 64 + k * 4 + c];
                    }
}

}  // namespace neo

using namespace neo;

namespace {

constexpr long kMaxElems = std::numeric_limits<int>::max();

bool valid_block(int b) {
    return b == 0 || b == 1 || b == 2 || b == 4 || b == 8 || b == 16 || b == 32 || b == 64;
}

long blocked_elems(long N, long C, long H, long W, int blk) {
    return blk ? N * ((C + blk - 1) / blk) * blk * H * W : N * C * H * W;
}

#define CHECK_PTR(p)                                                                        \
    do {                                                                                    \
        if (!(p)) return fail(NEO_ERR_INVALID_ARG, std::string(__func__) + ": " #p " is NULL"); \
        if (!aligned16(p))                                                                  \
            return fail(NEO_ERR_ALIGN, std::string(__func__) + ": " #p " not 16-byte aligned"); \
    } while (0)

#define CHECK_POS(v)                                                                       \
    do {                                                                                   \
        if ((v) <= 0)                                                                      \
            return fail(NEO_ERR_INVALID_ARG, std::string(__func__) + ": " #v " must be > 0"); \
    } while (0)

#define CHECK_SIZE(e)                                                                       \
    do {                                                                                    \
        if ((e) > kMaxElems)                                                                \
            return fail(NEO_ERR_UNSUPPORTED,                                                \
                        std::string(__func__) + ": tensor exceeds 2^31-1 elements");       \
    } while (0)

int out_dim(int n, int k, int s, int p) { return (n + 2 * p - k) / s + 1; }

// Split-reduction workspace of the standalone convolution call, one per
// (device, stream) so that calls on different streams never share it; calls
// on one stream are ordered by the stream.  Grows on demand (hipFree of the
// old buffer, hipMalloc of the new one); a call that would grow it while the
// stream is being captured into a graph fails with NEO_ERR_STATE and launches
// nothing (allocation is not capturable), so the first call of a given size
// must be made outside capture.
struct StreamWs {
    float* ws = nullptr;
    size_t bytes = 0;
};
std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, StreamWs> g_ws;

int stream_workspace(hipStream_t st, size_t bytes, float** ws) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "neo_conv2d_blocked: hipGetDevice");
    std::lock_guard<std::mutex> lk(g_ws_mu);
    StreamWs& w = g_ws[{dev, st}];
    if (w.bytes < bytes) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        e = hipStreamIsCapturing(st, &cap);
        if (e != hipSuccess) return hip_fail(e, "neo_conv2d_blocked: hipStreamIsCapturing");
        if (cap != hipStreamCaptureStatusNone)
            return fail(NEO_ERR_STATE, "neo_conv2d_blocked: the split-reduction workspace must "
                                       "grow to " + std::to_string(bytes) + " bytes, which "
                                       "cannot happen during stream capture; make one call of "
                                       "this size outside capture first");
        if (w.ws) {
            e = hipFree(w.ws);
            w.ws = nullptr;
            w.bytes = 0;
            if (e != hipSuccess) return hip_fail(e, "neo_conv2d_blocked: hipFree of the workspace");
        }
        e = hipMalloc(&w.ws, bytes);
        if (e != hipSuccess) {
            w.ws = nullptr;
            return fail(NEO_ERR_OOM, std::string("neo_conv2d_blocked: workspace allocation of ") +
                                         std::to_string(bytes) + " bytes: " + hipGetErrorString(e));
        }
        w.bytes = bytes;
    }
    *ws = w.ws;
    return NEO_OK;
}

// Optional override of the launch configuration, "fk,fp,split[,waves]", for
// tuning sweeps of the standalone call.
bool env_config(ConvConfig* c) {
    const char* v = std::getenv("NEO_CONV_CONFIG");
    if (!v || !*v) return false;
    ConvConfig t{1, 1, 1, 4};
    const int n = std::sscanf(v, "%d,%d,%d,%d", &t.fk, &t.fp, &t.split, &t.waves);
    if (n < 3 || !conv_config_valid(t)) return false;
    *c = t;
    return true;
}

// Optional override of the Winograd launch configuration, "fk,fp,split,waves".
bool env_wino_config(const ConvShape& s, ConvConfig* c) {
    const char* v = std::getenv("NEO_WINO_CONFIG");
    if (!v || !*v) return false;
    ConvConfig t{1, 1, 1, 1};
    if (std::sscanf(v, "%d,%d,%d,%d", &t.fk, &t.fp, &t.split, &t.waves) != 4 ||
        !wino_config_valid(s, t))
        return false;
    *c = t;
    return true;
}

// Optional override of the INT8 launch configuration, "fk,fp,waves".
bool env_i8_config(const ConvShape& s, ConvConfig* c) {
    const char* v = std::getenv("NEO_I8_CONFIG");
    if (!v || !*v) return false;
    ConvConfig t{1, 1, 1, 1};
    if (std::sscanf(v, "%d,%d,%d", &t.fk, &t.fp, &t.waves) != 3 || !int8_config_valid(s, t))
        return false;
    *c = t;
    return true;
}

// Largest C * R * S whose exact int32 sum of products of values in
// [-127, 127] cannot overflow: 127^2 * 133,000 < 2^31.
constexpr long kMaxI8Reduction = 133000;

}  // namespace

namespace neo {

int conv_prepare(const char* fn, const float* x, int x_block, int N, int C, int H, int W,
                 const float* w_packed, int K, int R, int S, const float* bias, int stride_h,
                 int stride_w, int pad_h, int pad_w, const neo_epilogue* ep, const float* y,
                 int y_block, int y_blk_offset, int y_blk_total, ConvShape* shape,
                 ConvConfig* config, const float** residual) {
    const std::string f(fn);
    auto ptr_ok = [&](const void* p, const char* name) {
        if (!p) return fail(NEO_ERR_INVALID_ARG, f + ": " + name + " is NULL");
        if (!aligned16(p)) return fail(NEO_ERR_ALIGN, f + ": " + name + " not 16-byte aligned");
        return (int)NEO_OK;
    };
    int rc;
    if ((rc = ptr_ok(x, "x")) != NEO_OK || (rc = ptr_ok(w_packed, "w_packed")) != NEO_OK ||
        (rc = ptr_ok(y, "y")) != NEO_OK || (bias && (rc = ptr_ok(bias, "bias")) != NEO_OK))
        return rc;
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || K <= 0 || R <= 0 || S <= 0 || stride_h <= 0 ||
        stride_w <= 0)
        return fail(NEO_ERR_INVALID_ARG, f + ": sizes and strides must be > 0");
    if (pad_h < 0 || pad_w < 0) return fail(NEO_ERR_INVALID_ARG, f + ": negative pad");
    const int act = ep ? ep->act : NEO_ACT_NONE;
    if (act != NEO_ACT_NONE && act != NEO_ACT_RELU)
        return fail(NEO_ERR_INVALID_ARG, f + ": unknown activation");
    const float* res = ep ? ep->residual : nullptr;
    if (res && (rc = ptr_ok(res, "residual")) != NEO_OK) return rc;
    const int OH = out_dim(H, R, stride_h, pad_h), OW = out_dim(W, S, stride_w, pad_w);
    if (H + 2 * pad_h < R || W + 2 * pad_w < S || OH < 1 || OW < 1)
        return fail(NEO_ERR_SHAPE, f + ": empty output (window larger than padded input)");
    ConvShape s{N, C, H, W, K, R, S, stride_h, stride_w, pad_h, pad_w, OH, OW,
                y_blk_offset, y_blk_total, act};
    s.xb = x_block;
    s.yb = y_block;
    if (!conv_blocks_valid(s))
        return fail(NEO_ERR_UNSUPPORTED, f + ": blocks must be 16, 32 or 64 "
                                             "(input 1, 4 or 8 too when C <= 4)");
    const int KY = cdiv(K, y_block);
    if (y_blk_offset < 0 || y_blk_total < KY || y_blk_offset + KY > y_blk_total)
        return fail(NEO_ERR_SHAPE, f + ": output channel-block view out of range");
    if (blocked_elems(N, C, H, W, x_block) > kMaxElems ||
        (long)N * y_blk_total * y_block * OH * OW > kMaxElems ||
        (long)cdiv(K, 16) * 16 * cdiv(C, 16) * 16 * R * S > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, f + ": tensor exceeds 2^31-1 elements");
    if (blocked_elems(N, C, H, W, x_block) >= (1L << 29) ||
        (long)cdiv(K, 16) * cdiv(C, 16) * R * S * 256 >= (1L << 29))
        return fail(NEO_ERR_UNSUPPORTED, f + ": input or filter of 2 GiB or more");
    ConvConfig cfg = choose_conv_config(s);
    (void)tuned_config(s, false, &cfg);
    env_config(&cfg);
    const int T = cdiv(C, 16) * R * S;
    if (cfg.split > T) cfg.split = T;
    *shape = s;
    *config = cfg;
    *residual = res;
    return NEO_OK;
}

}  // namespace neo

namespace {

int conv_int8_common(const char* fn, const int8_t* xq, int N, int C, int H, int W,
                     const int8_t* w_packed, const float* w_scale, int K, int R, int S,
                     float x_scale, const float* bias, int stride_h, int stride_w, int pad_h,
                     int pad_w, const neo_epilogue* ep, float* y, int y_cblk_offset,
                     int y_cblk_total, int* acc, int8_t* yq, float y_scale, int y_pad_h,
                     int y_pad_w, neo_stream_t stream) {
    const std::string f(fn);
    float* out = acc ? reinterpret_cast<float*>(acc) : yq ? reinterpret_cast<float*>(yq) : y;
    ConvShape s;
    ConvConfig cfg;
    const float* res = nullptr;
    // the shape, view and pointer checks of the fp32 convolution (an int8
    // tensor is a quarter of the fp32 one's bytes, so its limits hold too)
    int rc = conv_prepare(fn, reinterpret_cast<const float*>(xq), 16, N, C, H, W,
                          reinterpret_cast<const float*>(w_packed), K, R, S, bias, stride_h,
                          stride_w, pad_h, pad_w, ep, out, 16, y_cblk_offset, y_cblk_total, &s,
                          &cfg, &res);
    if (rc != NEO_OK) return rc;
    if (!acc) {
        if (!w_scale) return fail(NEO_ERR_INVALID_ARG, f + ": w_scale is NULL");
        if (!aligned16(w_scale)) return fail(NEO_ERR_ALIGN, f + ": w_scale not 16-byte aligned");
        if (!(x_scale > 0.f) || !std::isfinite(x_scale))
            return fail(NEO_ERR_INVALID_ARG, f + ": x_scale must be finite and > 0");
    }
    if (yq) {
        if (!(y_scale > 0.f) || !std::isfinite(y_scale) || !std::isfinite(1.0f / y_scale))
            return fail(NEO_ERR_INVALID_ARG, f + ": y_scale must be finite, > 0 and have a "
                                                 "finite reciprocal");
        if (y_pad_h < 0 || y_pad_w < 0) return fail(NEO_ERR_INVALID_ARG, f + ": negative y pad");
        if ((long)N * y_cblk_total * (s.OH + 2L * y_pad_h) * (s.OW + 2L * y_pad_w) * 16 > kMaxElems)
            return fail(NEO_ERR_UNSUPPORTED, f + ": padded int8 output of 2 GiB or more");
    }
    if ((long)C * R * S > kMaxI8Reduction)
        return fail(NEO_ERR_UNSUPPORTED, f + ": C * R * S above 133,000 could overflow the "
                                             "int32 accumulator");
    if (int8_filter_bytes(K, C, R, S) > (size_t)kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, f + ": packed filter of 2 GiB or more");
    // (four channel-block planes of slack: the loads of blocks past the last
    // stay below 2^31 as byte offsets and read 0 through the range check)
    if (((long)N * cdiv(C, 16) + 4) * (H + 2L * pad_h) * (W + 2L * pad_w) * 16 > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, f + ": padded int8 input of 2 GiB or more");
    cfg = choose_int8_config(s);
    if (!acc) (void)tuned_int8_config(s, yq ? 2 : 0, &cfg);
    env_i8_config(s, &cfg);
    hipError_t e = launch_conv_int8(s, cfg, xq, w_packed, w_scale, x_scale, bias, res, y, acc, yq,
                                    y_scale, y_pad_h, y_pad_w, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, (f + " launch").c_str());
}

}  // namespace

extern "C" {

const char* neo_last_error(void) { return g_err.c_str(); }

int neo_conv2d_nchwxc(const float* x, int x_block, int N, int C, int H, int W,
                      const float* w_packed, int K, int R, int S, const float* bias, int stride_h,
                      int stride_w, int pad_h, int pad_w, const neo_epilogue* ep, float* y,
                      int y_block, int y_blk_offset, int y_blk_total, neo_stream_t stream) {
    ConvShape s;
    ConvConfig cfg;
    const float* res = nullptr;
    int rc = conv_prepare("neo_conv2d_nchwxc", x, x_block, N, C, H, W, w_packed, K, R, S, bias,
                          stride_h, stride_w, pad_h, pad_w, ep, y, y_block, y_blk_offset,
                          y_blk_total, &s, &cfg, &res);
    if (rc != NEO_OK) return rc;
    float* ws = nullptr;
    if (cfg.split > 1) {
        rc = stream_workspace((hipStream_t)stream, conv_workspace_bytes(s, cfg), &ws);
        if (rc != NEO_OK) return rc;
    }
    hipError_t e = launch_conv2d(s, cfg, x, w_packed, false, bias, res, y, ws,
                                 (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_conv2d_nchwxc launch");
}

int neo_conv2d_blocked(const float* x, int N, int C, int H, int W, const float* w_packed, int K,
                       int R, int S, const float* bias, int stride_h, int stride_w, int pad_h,
                       int pad_w, const neo_epilogue* ep, float* y, int y_cblk_offset,
                       int y_cblk_total, neo_stream_t stream) {
    return neo_conv2d_nchwxc(x, 16, N, C, H, W, w_packed, K, R, S, bias, stride_h, stride_w, pad_h,
                             pad_w, ep, y, 16, y_cblk_offset, y_cblk_total, stream);
}

int neo_layout_transform(const float* src, int src_block, float* dst, int dst_block, int N,
                         int C, int H, int W, neo_stream_t stream) {
    if (!src || !dst) return fail(NEO_ERR_INVALID_ARG, "neo_layout_transform: NULL buffer");
    if (!valid_block(src_block) || !valid_block(dst_block))
        return fail(NEO_ERR_INVALID_ARG, "neo_layout_transform: block must be 0,1,2,4,8,16,32,64");
    CHECK_POS(N); CHECK_POS(C); CHECK_POS(H); CHECK_POS(W);
    if ((src_block >= 4 || dst_block >= 4) && (!aligned16(src) || !aligned16(dst)))
        return fail(NEO_ERR_ALIGN, "neo_layout_transform: buffers not 16-byte aligned");
    CHECK_SIZE(blocked_elems(N, C, H, W, src_block));
    CHECK_SIZE(blocked_elems(N, C, H, W, dst_block));
    const long sb = blocked_elems(N, C, H, W, src_block) * 4, db = blocked_elems(N, C, H, W, dst_block) * 4;
    const char* s0 = (const char*)src;
    const char* d0 = (const char*)dst;
    if (s0 < d0 + db && d0 < s0 + sb)
        return fail(NEO_ERR_INVALID_ARG, "neo_layout_transform: src and dst overlap");
    hipError_t e = launch_layout_transform(src, src_block, dst, dst_block, N, C, H, W, 0,
                                           dst_block ? cdiv(C, dst_block) : C, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_layout_transform launch");
}

int neo_pack_filter(const float* w_kcrs, int K, int C, int R, int S, int ic_bn, int oc_bn,
                    float* w_packed, neo_stream_t stream) {
    if (!w_kcrs || !w_packed) return fail(NEO_ERR_INVALID_ARG, "neo_pack_filter: NULL buffer");
    CHECK_POS(K); CHECK_POS(C); CHECK_POS(R); CHECK_POS(S);
    if (!valid_block(ic_bn) || !valid_block(oc_bn) || ic_bn == 0 || oc_bn == 0)
        return fail(NEO_ERR_INVALID_ARG, "neo_pack_filter: ic_bn/oc_bn must be 1,2,4,8,16,32,64");
    CHECK_SIZE((long)cdiv(K, oc_bn) * oc_bn * cdiv(C, ic_bn) * ic_bn * R * S);
    hipError_t e = launch_pack_filter(w_kcrs, K, C, R, S, ic_bn, oc_bn, w_packed, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_pack_filter launch");
}

int neo_winograd_filter(const float* w_kcrs, int K, int C, float* u, neo_stream_t stream) {
    if (!w_kcrs || !u) return fail(NEO_ERR_INVALID_ARG, "neo_winograd_filter: NULL buffer");
    CHECK_POS(K); CHECK_POS(C);
    if ((long)cdiv(K, 16) * cdiv(C, 16) * 16 * 256 >= (1L << 29))
        return fail(NEO_ERR_UNSUPPORTED, "neo_winograd_filter: transformed filter of 2 GiB or more");
    hipError_t e = launch_wino_filter(w_kcrs, K, C, u, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_winograd_filter launch");
}

int neo_conv2d_winograd(const float* x, int N, int C, int H, int W, const float* u, int K,
                        const float* bias, int pad_h, int pad_w, const neo_epilogue* ep, float* y,
                        int y_cblk_offset, int y_cblk_total, neo_stream_t stream) {
    ConvShape s;
    ConvConfig cfg;
    const float* res = nullptr;
    int rc = conv_prepare("neo_conv2d_winograd", x, 16, N, C, H, W, u, K, 3, 3, bias, 1, 1, pad_h,
                          pad_w, ep, y, 16, y_cblk_offset, y_cblk_total, &s, &cfg, &res);
    if (rc != NEO_OK) return rc;
    if (conv_small_c(s))
        return fail(NEO_ERR_UNSUPPORTED, "neo_conv2d_winograd: needs more than 4 input channels "
                                         "(use neo_conv2d_blocked)");
    if (wino_filter_floats(s) >= (1UL << 29))
        return fail(NEO_ERR_UNSUPPORTED, "neo_conv2d_winograd: transformed filter of 2 GiB or more");
    cfg = choose_wino_config(s);
    env_wino_config(s, &cfg);
    float* ws = nullptr;
    if (cfg.split > 1) {
        rc = stream_workspace((hipStream_t)stream, conv_workspace_bytes(s, cfg), &ws);
        if (rc != NEO_OK) return rc;
    }
    hipError_t e = launch_wino(s, cfg, x, u, bias, res, y, ws, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_conv2d_winograd launch");
}

int neo_quantize_int8(const float* x, int N, int C, int H, int W, float x_scale, int pad_h,
                      int pad_w, int8_t* xq, neo_stream_t stream) {
    if (!x || !xq) return fail(NEO_ERR_INVALID_ARG, "neo_quantize_int8: NULL buffer");
    if (!aligned16(x) || !aligned16(xq))
        return fail(NEO_ERR_ALIGN, "neo_quantize_int8: buffers not 16-byte aligned");
    CHECK_POS(N); CHECK_POS(C); CHECK_POS(H); CHECK_POS(W);
    if (pad_h < 0 || pad_w < 0) return fail(NEO_ERR_INVALID_ARG, "neo_quantize_int8: negative pad");
    if (!(x_scale > 0.f) || !std::isfinite(x_scale))
        return fail(NEO_ERR_INVALID_ARG, "neo_quantize_int8: x_scale must be finite and > 0");
    CHECK_SIZE(blocked_elems(N, C, H, W, 16));
    if ((long)N * cdiv(C, 16) * (H + 2L * pad_h) * (W + 2L * pad_w) * 16 > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, "neo_quantize_int8: padded int8 tensor of 2 GiB or more");
    hipError_t e = launch_quantize_int8(x, N, C, H, W, pad_h, pad_w, x_scale, xq, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_quantize_int8 launch");
}

int neo_pack_filter_int8(const float* w_kcrs, int K, int C, int R, int S, int8_t* w_packed,
                         float* w_scale, neo_stream_t stream) {
    if (!w_kcrs || !w_packed || !w_scale)
        return fail(NEO_ERR_INVALID_ARG, "neo_pack_filter_int8: NULL buffer");
    CHECK_POS(K); CHECK_POS(C); CHECK_POS(R); CHECK_POS(S);
    CHECK_SIZE((long)K * C * R * S);
    if (int8_filter_bytes(K, C, R, S) > (size_t)kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, "neo_pack_filter_int8: packed filter of 2 GiB or more");
    hipError_t e = launch_pack_filter_int8(w_kcrs, K, C, R, S, w_packed, w_scale, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_pack_filter_int8 launch");
}

int neo_conv2d_int8(const int8_t* xq, int N, int C, int H, int W, const int8_t* w_packed,
                    const float* w_scale, int K, int R, int S, float x_scale, const float* bias,
                    int stride_h, int stride_w, int pad_h, int pad_w, const neo_epilogue* ep,
                    float* y, int y_cblk_offset, int y_cblk_total, neo_stream_t stream) {
    return conv_int8_common("neo_conv2d_int8", xq, N, C, H, W, w_packed, w_scale, K, R, S, x_scale,
                            bias, stride_h, stride_w, pad_h, pad_w, ep, y, y_cblk_offset,
                            y_cblk_total, nullptr, nullptr, 0.f, 0, 0, stream);
}

int neo_conv2d_int8_q(const int8_t* xq, int N, int C, int H, int W, const int8_t* w_packed,
                      const float* w_scale, int K, int R, int S, float x_scale, const float* bias,
                      int stride_h, int stride_w, int pad_h, int pad_w, const neo_epilogue* ep,
                      float y_scale, int y_pad_h, int y_pad_w, int8_t* yq, int y_cblk_offset,
                      int y_cblk_total, neo_stream_t stream) {
    if (!yq) return fail(NEO_ERR_INVALID_ARG, "neo_conv2d_int8_q: yq is NULL");
    return conv_int8_common("neo_conv2d_int8_q", xq, N, C, H, W, w_packed, w_scale, K, R, S,
                            x_scale, bias, stride_h, stride_w, pad_h, pad_w, ep, nullptr,
                            y_cblk_offset, y_cblk_total, nullptr, yq, y_scale, y_pad_h, y_pad_w,
                            stream);
}

int neo_conv2d_int8_acc(const int8_t* xq, int N, int C, int H, int W, const int8_t* w_packed, int K,
                        int R, int S, int stride_h, int stride_w, int pad_h, int pad_w, int32_t* acc,
                        neo_stream_t stream) {
    if (!acc) return fail(NEO_ERR_INVALID_ARG, "neo_conv2d_int8_acc: acc is NULL");
    return conv_int8_common("neo_conv2d_int8_acc", xq, N, C, H, W, w_packed, nullptr, K, R, S, 1.f,
                            nullptr, stride_h, stride_w, pad_h, pad_w, nullptr, nullptr, 0,
                            cdiv(K, 16), acc, nullptr, 0.f, 0, 0, stream);
}

int neo_pack_dense_int8(const float* w, int out_features, int in_features, int8_t* w_rows, float* w_scale,
                        neo_stream_t stream) {
    if (!w || !w_rows || !w_scale) return fail(NEO_ERR_INVALID_ARG, "neo_pack_dense_int8: NULL buffer");
    if (!aligned16(w_rows)) return fail(NEO_ERR_ALIGN, "neo_pack_dense_int8: w_rows not 16-byte aligned");
    CHECK_POS(out_features); CHECK_POS(in_features);
    CHECK_SIZE((long)out_features * in_features);
    if ((long)out_features * (long)dense_i8_row_bytes(in_features) > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, "neo_pack_dense_int8: int8 weights of 2 GiB or more");
    hipError_t e = launch_pack_dense_int8(w, out_features, in_features, w_rows, w_scale, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_pack_dense_int8 launch");
}

int neo_quantize_rows_int8(const float* x, int N, int in_features, float x_scale, int8_t* xq,
                           neo_stream_t stream) {
    if (!x || !xq) return fail(NEO_ERR_INVALID_ARG, "neo_quantize_rows_int8: NULL buffer");
    if (!aligned16(xq)) return fail(NEO_ERR_ALIGN, "neo_quantize_rows_int8: xq not 16-byte aligned");
    CHECK_POS(N); CHECK_POS(in_features);
    if (!(x_scale > 0.f) || !std::isfinite(x_scale))
        return fail(NEO_ERR_INVALID_ARG, "neo_quantize_rows_int8: x_scale must be finite and > 0");
    if ((long)N * (long)dense_i8_row_bytes(in_features) > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, "neo_quantize_rows_int8: rows of 2 GiB or more");
    hipError_t e = launch_quantize_rows_int8(x, N, in_features, x_scale, xq, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_quantize_rows_int8 launch");
}

int neo_dense_int8(const int8_t* xq, int N, int in_features, const int8_t* w_rows, const float* w_scale,
                   int out_features, float x_scale, const float* bias, int act, float* y, float y_scale,
                   int8_t* yq, neo_stream_t stream) {
    if (!xq || !w_rows || !w_scale) return fail(NEO_ERR_INVALID_ARG, "neo_dense_int8: NULL buffer");
    if (!y && !yq) return fail(NEO_ERR_INVALID_ARG, "neo_dense_int8: neither y nor yq given");
    if (!aligned16(xq) || !aligned16(w_rows))
        return fail(NEO_ERR_ALIGN, "neo_dense_int8: xq and w_rows must be 16-byte aligned");
    CHECK_POS(N); CHECK_POS(in_features); CHECK_POS(out_features);
    if (act != NEO_ACT_NONE && act != NEO_ACT_RELU) return fail(NEO_ERR_INVALID_ARG, "neo_dense_int8: act");
    if (!(x_scale > 0.f) || !std::isfinite(x_scale))
        return fail(NEO_ERR_INVALID_ARG, "neo_dense_int8: x_scale must be finite and > 0");
    if (yq && (!(y_scale > 0.f) || !std::isfinite(y_scale) || !std::isfinite(1.0f / y_scale)))
        return fail(NEO_ERR_INVALID_ARG, "neo_dense_int8: y_scale must be finite, > 0, with a finite reciprocal");
    if ((long)in_features * 127 * 127 >= (1L << 31))
        return fail(NEO_ERR_UNSUPPORTED, "neo_dense_int8: in_features above 133,144 could overflow int32");
    if ((long)N * (long)dense_i8_row_bytes(in_features) > kMaxElems ||
        (long)out_features * (long)dense_i8_row_bytes(in_features) > kMaxElems ||
        (long)N * out_features > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, "neo_dense_int8: a tensor of 2 GiB or more");
    hipError_t e = launch_dense_int8(xq, w_rows, w_scale, x_scale, bias, N, in_features, out_features, act, y, yq,
                                     y_scale, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_dense_int8 launch");
}

int neo_fold_bn(const float* w, const float* bias, const float* gamma, const float* beta,
                const float* mean, const float* var, float eps, int K, int C, int R, int S,
                float* w_out, float* bias_out) {
    if (!w || !gamma || !beta || !mean || !var || !w_out || !bias_out)
        return fail(NEO_ERR_INVALID_ARG, "neo_fold_bn: NULL pointer");
    CHECK_POS(K); CHECK_POS(C); CHECK_POS(R); CHECK_POS(S);
    if (!(eps >= 0.f)) return fail(NEO_ERR_INVALID_ARG, "neo_fold_bn: eps must be >= 0");
    for (int k = 0; k < K; ++k)
        if (!((double)var[k] + (double)eps > 0.0))
            return fail(NEO_ERR_INVALID_ARG, "neo_fold_bn: var + eps must be > 0");
    fold_bn_host(w, bias, gamma, beta, mean, var, eps, K, C, R, S, w_out, bias_out);
    return NEO_OK;
}

static int pool_common(const char* fn, bool is_max, const float* x, int blk, int N, int C, int H,
                       int W, int R, int S, int sh, int sw, int ph, int pw, float* y, int y_off,
                       int y_tot, neo_stream_t stream) {
    if (!x || !y) return fail(NEO_ERR_INVALID_ARG, std::string(fn) + ": NULL buffer");
    if (!aligned16(x) || !aligned16(y)) return fail(NEO_ERR_ALIGN, std::string(fn) + ": unaligned buffer");
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0 || R <= 0 || S <= 0 || sh <= 0 || sw <= 0 || ph < 0 ||
        pw < 0)
        return fail(NEO_ERR_INVALID_ARG, std::string(fn) + ": non-positive size");
    if (ph >= R || pw >= S) return fail(NEO_ERR_INVALID_ARG, std::string(fn) + ": pad must be < window");
    const int OH = out_dim(H, R, sh, ph), OW = out_dim(W, S, sw, pw);
    if (H + 2 * ph < R || W + 2 * pw < S || OH < 1 || OW < 1)
        return fail(NEO_ERR_SHAPE, std::string(fn) + ": empty output");
    if (!pow2_block(blk))
        return fail(NEO_ERR_UNSUPPORTED, std::string(fn) + ": block must be 4, 8, 16, 32 or 64");
    const int CB = cdiv(C, blk);
    if (y_off < 0 || y_off + CB > y_tot)
        return fail(NEO_ERR_SHAPE, std::string(fn) + ": output channel-block view out of range");
    if (blocked_elems(N, C, H, W, blk) > kMaxElems || (long)N * y_tot * blk * OH * OW > kMaxElems)
        return fail(NEO_ERR_UNSUPPORTED, std::string(fn) + ": tensor exceeds 2^31-1 elements");
    PoolShape s{N, C, H, W, R, S, sh, sw, ph, pw, OH, OW, y_off, y_tot};
    s.xb = blk;
    hipError_t e = is_max ? launch_maxpool(s, x, y, (hipStream_t)stream)
                          : launch_avgpool(s, x, y, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, fn);
}

int neo_maxpool2d_blocked(const float* x, int N, int C, int H, int W, int R, int S, int stride_h,
                          int stride_w, int pad_h, int pad_w, float* y, int y_cblk_offset,
                          int y_cblk_total, neo_stream_t stream) {
    return pool_common("neo_maxpool2d_blocked", true, x, 16, N, C, H, W, R, S, stride_h, stride_w,
                       pad_h, pad_w, y, y_cblk_offset, y_cblk_total, stream);
}

int neo_avgpool2d_blocked(const float* x, int N, int C, int H, int W, int R, int S, int stride_h,
                          int stride_w, int pad_h, int pad_w, float* y, int y_cblk_offset,
                          int y_cblk_total, neo_stream_t stream) {
    return pool_common("neo_avgpool2d_blocked", false, x, 16, N, C, H, W, R, S, stride_h, stride_w,
                       pad_h, pad_w, y, y_cblk_offset, y_cblk_total, stream);
}

int neo_maxpool2d_nchwxc(const float* x, int block, int N, int C, int H, int W, int R, int S,
                         int stride_h, int stride_w, int pad_h, int pad_w, float* y,
                         int y_blk_offset, int y_blk_total, neo_stream_t stream) {
    return pool_common("neo_maxpool2d_nchwxc", true, x, block, N, C, H, W, R, S, stride_h,
                       stride_w, pad_h, pad_w, y, y_blk_offset, y_blk_total, stream);
}

int neo_avgpool2d_nchwxc(const float* x, int block, int N, int C, int H, int W, int R, int S,
                         int stride_h, int stride_w, int pad_h, int pad_w, float* y,
                         int y_blk_offset, int y_blk_total, neo_stream_t stream) {
    return pool_common("neo_avgpool2d_nchwxc", false, x, block, N, C, H, W, R, S, stride_h,
                       stride_w, pad_h, pad_w, y, y_blk_offset, y_blk_total, stream);
}

int neo_global_avgpool_nchwxc(const float* x, int block, int N, int C, int H, int W, float* y,
                              neo_stream_t stream) {
    CHECK_PTR(x);
    CHECK_PTR(y);
    CHECK_POS(N); CHECK_POS(C); CHECK_POS(H); CHECK_POS(W);
    if (!pow2_block(block))
        return fail(NEO_ERR_UNSUPPORTED, "neo_global_avgpool_nchwxc: block must be 4, 8, 16, 32 or 64");
    CHECK_SIZE(blocked_elems(N, C, H, W, block));
    hipError_t e = launch_gap(x, block, N, C, H, W, y, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_global_avgpool_nchwxc launch");
}

int neo_global_avgpool_blocked(const float* x, int N, int C, int H, int W, float* y,
                               neo_stream_t stream) {
    return neo_global_avgpool_nchwxc(x, 16, N, C, H, W, y, stream);
}

int neo_dense(const float* x, int N, int IN, const float* w, int OUT, const float* bias, int act,
              float* y, neo_stream_t stream) {
    if (!x || !w || !y) return fail(NEO_ERR_INVALID_ARG, "neo_dense: NULL buffer");
    CHECK_POS(N); CHECK_POS(IN); CHECK_POS(OUT);
    if (act != NEO_ACT_NONE && act != NEO_ACT_RELU)
        return fail(NEO_ERR_INVALID_ARG, "neo_dense: unknown activation");
    CHECK_SIZE((long)N * IN);
    CHECK_SIZE((long)OUT * IN);
    CHECK_SIZE((long)N * OUT);
    hipError_t e = launch_dense(x, N, IN, w, OUT, bias, act, y, (hipStream_t)stream);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_dense launch");
}

}  // extern "C"
