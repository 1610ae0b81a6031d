// Pointwise convolutions with few input channels as a stream: each wave keeps
// its output channels' filter in registers and walks a strided sequence of
// 16-pixel groups, the next groups' inputs (and residuals) loading while it
// multiplies the current one.
//
// A 1x1 conv over 64 input channels at batch 32 (ResNet-50's 64 -> 64 and
// 64 -> 256 layers at 56x56) does 4 reduction steps per 16x16 tile, so the
// tile kernel's waves spend their life waiting for their first operands and
// their stores: the layer is bound by how many bytes are in flight, not by
// MFMAs.  Here a wave loads its filter blocks (fk output blocks x CB input
// blocks, one float4 per lane and MFMA k-quad) once, then for every pixel
// group: the lane's input float4 of each input block, 4 x fk x CB MFMAs, and
// act(acc + bias + residual) stored as one float4 per output block.  DEPTH
// groups are in flight per wave.
// The per-output sum runs over the input blocks in order, each block's four
// k-steps in order: the tile kernel's order with one wave and no split, so the
// results are bit-identical to it.
#include "conv_kernel.h"

namespace neo {

using conv_detail::FastDiv;
using conv_detail::fdiv;
using conv_detail::make_fastdiv;
using conv_detail::v4f;

namespace {

struct StreamArgs {
    const float* x;     // NCHW16c input, CB blocks
    const float* w;     // kernel filter order: block (kb, cb) = 64 lane float4s
    const float* bias;  // [KB * 16] or null
    const float* res;   // NCHW16c, KB blocks, or null
    float* y;           // NCHW16c view: blocks [y_off, y_off + KB) of y_tot
    int CB, KB, OHW, M, groups, act, y_off, y_tot;
    int nkt;            // channel tiles (KB / FK)
    int waves_per_kt;   // waves walking the pixel groups of one channel tile
    FastDiv div_ohw;
};

template <int FK, int CBMAX, int DEPTH>
__global__ __launch_bounds__(256) void conv1x1_stream(StreamArgs a) {
    const int lane = threadIdx.x & 63;
    const int li = lane & 15, g = lane >> 4;
    const int gw = __builtin_amdgcn_readfirstlane((int)(blockIdx.x * 4 + (threadIdx.x >> 6)));
    // consecutive waves take consecutive channel tiles of one pixel group, so
    // the waves that read one input group run together on one XCD
    const int kt = gw % a.nkt;
    const int j0 = gw / a.nkt;
    if (j0 >= a.waves_per_kt) return;
    const int kb0 = kt * FK;

    v4f wa[FK][CBMAX];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int cb = 0; cb < CBMAX; ++cb)
            wa[f][cb] = cb < a.CB ? *reinterpret_cast<const v4f*>(
                                        a.w + (((long)(kb0 + f) * a.CB + cb) * 64 + g * 16 + li) * 4)
                                  : v4f{0.f, 0.f, 0.f, 0.f};
    v4f bb[FK];
#pragma unroll
    for (int f = 0; f < FK; ++f)
        bb[f] = a.bias ? *reinterpret_cast<const v4f*>(a.bias + (kb0 + f) * 16 + 4 * g)
                       : v4f{0.f, 0.f, 0.f, 0.f};

    // pixel group q of this wave's sequence: q-th group j0 + q * waves_per_kt
    struct Slot {
        v4f x[CBMAX];
        v4f r[FK];
        int n, pix;
        bool ok;
    };
    auto load = [&](Slot& s, int grp) {
        const int m = grp * 16 + li;
        s.ok = grp < a.groups && m < a.M;
        const int mm = s.ok ? m : 0;
        s.n = fdiv(mm, a.div_ohw);
        s.pix = mm - s.n * a.OHW;
#pragma unroll
        for (int cb = 0; cb < CBMAX; ++cb)
            if (cb < a.CB)
                s.x[cb] = *reinterpret_cast<const v4f*>(
                    a.x + (((long)s.n * a.CB + cb) * a.OHW + s.pix) * 16 + 4 * g);
#pragma unroll
        for (int f = 0; f < FK; ++f)
            s.r[f] = a.res ? *reinterpret_cast<const v4f*>(
                                 a.res + (((long)s.n * a.KB + kb0 + f) * a.OHW + s.pix) * 16 + 4 * g)
                           : v4f{0.f, 0.f, 0.f, 0.f};
    };
    // ring[d] holds group grp + d * waves_per_kt; a slot is refilled with the
    // group DEPTH steps further once its epilogue has read it, so DEPTH - 1
    // groups are in flight while one is multiplied
    Slot ring[DEPTH];
#pragma unroll
    for (int d = 0; d < DEPTH; ++d) load(ring[d], j0 + d * a.waves_per_kt);
    for (int grp = j0; grp < a.groups; grp += DEPTH * a.waves_per_kt) {
#pragma unroll
        for (int d = 0; d < DEPTH; ++d) {
            const int cur = grp + d * a.waves_per_kt;
            if (cur >= a.groups) break;
            Slot& s = ring[d];
            v4f acc[FK];
#pragma unroll
            for (int f = 0; f < FK; ++f) acc[f] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int cb = 0; cb < CBMAX; ++cb) {
                if (cb >= a.CB) break;
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int f = 0; f < FK; ++f)
                        acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[f][cb][t], s.x[cb][t], acc[f], 0, 0, 0);
            }
            if (s.ok) {
#pragma unroll
                for (int f = 0; f < FK; ++f) {
                    v4f o = acc[f] + bb[f];
                    if (a.res) o += s.r[f];
                    if (a.act == NEO_ACT_RELU) {
#pragma unroll
                        for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
                    }
                    *reinterpret_cast<v4f*>(
                        a.y + (((long)s.n * a.y_tot + a.y_off + kb0 + f) * a.OHW + s.pix) * 16 + 4 * g) = o;
                }
            }
            load(s, cur + DEPTH * a.waves_per_kt);
        }
    }
}

constexpr int kDepth = 3;

template <int FK, int CBMAX>
hipError_t launch_t(const StreamArgs& a, int wgs, hipStream_t st) {
    hipLaunchKernelGGL((conv1x1_stream<FK, CBMAX, kDepth>), dim3(wgs), dim3(256), 0, st, a);
    return hipGetLastError();
}

}  // namespace

bool conv_stream_eligible(const ConvShape& s) {
    return s.R == 1 && s.S == 1 && s.sh == 1 && s.sw == 1 && s.ph == 0 && s.pw == 0 && s.xb == 16 &&
           s.yb == 16 && !s.gap && !conv_small_c(s) && cdiv(s.C, 16) <= 8;
}

bool conv_stream_config_valid(const ConvShape& s, const ConvConfig& c) {
    // the filter a wave holds: fk x CB float4s per lane, at most 16
    return conv_stream_eligible(s) && c.fp == 0 && c.split == 1 &&
           (c.fk == 1 || c.fk == 2 || c.fk == 4) && cdiv(s.K, 16) % c.fk == 0 &&
           c.fk * cdiv(s.C, 16) <= 16 &&
           (c.waves == 1 || c.waves == 2 || c.waves == 4 || c.waves == 8);
}

hipError_t launch_conv_stream(const ConvShape& s, const ConvConfig& c, const float* x, const float* w,
                              const float* bias, const float* res, float* y, hipStream_t st) {
    if (!conv_stream_config_valid(s, c)) return hipErrorInvalidValue;
    StreamArgs a;
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.res = res;
    a.y = y;
    a.CB = cdiv(s.C, 16);
    a.KB = cdiv(s.K, 16);
    a.OHW = s.OH * s.OW;
    a.M = s.N * a.OHW;
    a.groups = cdiv(a.M, 16);
    a.act = s.act;
    a.y_off = s.y_off;
    a.y_tot = s.y_tot;
    a.nkt = a.KB / c.fk;
    a.div_ohw = make_fastdiv((unsigned)a.OHW);
    // waves: c.waves per SIMD of the chip (1024 SIMDs), at most one per group
    // and channel tile
    const long total = std::min<long>((long)c.waves * 1024, (long)a.groups * a.nkt);
    a.waves_per_kt = (int)std::max<long>(1, total / a.nkt);
    const long wgs = cdiv((int)std::min<long>((long)a.waves_per_kt * a.nkt, 1L << 28), 4);
    const bool small = a.CB <= 4;
    switch (c.fk) {
        case 1: return small ? launch_t<1, 4>(a, (int)wgs, st) : launch_t<1, 8>(a, (int)wgs, st);
        case 2: return small ? launch_t<2, 4>(a, (int)wgs, st) : launch_t<2, 8>(a, (int)wgs, st);
        case 4: return small ? launch_t<4, 4>(a, (int)wgs, st) : hipErrorInvalidValue;
        default: return hipErrorInvalidValue;
    }
}

}  // namespace neo
