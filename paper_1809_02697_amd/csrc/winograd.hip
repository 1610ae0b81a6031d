// Winograd F(2x2, 3x3) convolution on fp32 MFMA (gfx950) -- the fast
// convolution algorithm the paper names as future work beside its direct
// convolution (Sections 1 and 5).  One launch per layer, NCHW16c in and out:
//
//   - A lane owns one 2x2 output tile (tile i of a 16-tile group) and the
//     channel quad 4g..4g+3 of the MFMA layout.  Per input channel block it
//     loads the tile's 4x4 patch (16 float4, zero outside the input through
//     the buffer range check, like the direct kernel's padding taps) and
//     applies B^T d B in registers: additions only.
//   - The 16 elements of the transformed tile are 16 independent products
//     over the input channels, M_e = U_e V_e: per channel block and element,
//     4 MFMA k-steps of v_mfma_f32_16x16x4f32 with the transformed filter
//     (16 output channels x 4 input channels, one float4 per lane, in the
//     same [c/4][k][c%4] order as the direct kernel's filter blocks) as the
//     A operand and the transformed input as B.  Accumulator register v of
//     lane (i, g) then holds M_e[k = 4g + v][tile i]: all 16 elements of one
//     (output channel, tile) sit in one lane.
//   - The waves of a workgroup take different tile groups and the same
//     output blocks, so they share the transformed filter: per channel block
//     the workgroup stages its FK x 16 KB in LDS (double-buffered, the next
//     block's loads in flight while this block's MFMAs run, one barrier per
//     block), and each wave reads its A operands from LDS.
//   - A^T M A (additions only) gives the 2x2 outputs in registers; then
//     act(y + bias + residual) and one float4 store per output pixel -- or,
//     when the channel blocks are split across workgroups, raw partial
//     outputs for the split reduction kernel the direct convolution uses (the
//     output transform is linear).
//
// A layer's multiplications fall from 9 to 4 per output: 16 MFMA k-step
// groups for a 2x2 tile instead of 9 per output pixel, i.e. 2.25x fewer MFMAs
// than the direct kernel, for the cost of the transforms and of a filter 16/9
// larger.  The rounding differs from the direct sum (the transforms add and
// cancel larger intermediate values), so results match the oracle within the
// tolerance but are not bit-identical to the direct kernel's.
#include "conv_kernel.h"
#include "winograd.h"

namespace neo {

using conv_detail::ConvArgs;
using conv_detail::FastDiv;
using conv_detail::fdiv;
using conv_detail::kOutOfRange;
using conv_detail::kRsrcWord3;
using conv_detail::ld4;
using conv_detail::make_fastdiv;
using conv_detail::v4f;
using conv_detail::xcd_order;

namespace {

struct WinoArgs {
    const float* x;     // NCHW16c [N][CB][H][W][16]
    const float* u;     // transformed filter [KB][CB][16][256]
    const float* bias;  // [KB * 16] or null
    const float* res;   // NCHW16c [N][KB][OH][OW][16] or null
    float* y;           // NCHW16c view: blocks [y_off, y_off + KB) of y_tot
    float* ws;          // split partials [split][N][KB][OH][OW][16]
    int N, CB, H, W, KB, OH, OW, ph, pw, TH, TW, NT, y_off, y_tot, act, split;
    int ntg, nkt;       // tile units of WAVES * FT * 16 tiles; channel tiles of FK blocks
    int x_bytes, u_bytes;
    FastDiv div_tt, div_tw;  // tiles per image, tiles per row
};

// The 1D input transform B^T applied to four values: (d0 - d2, d1 + d2,
// d2 - d1, d1 - d3).
__device__ inline void bt4(const v4f& d0, const v4f& d1, const v4f& d2, const v4f& d3, v4f& o0,
                           v4f& o1, v4f& o2, v4f& o3) {
    o0 = d0 - d2;
    o1 = d1 + d2;
    o2 = d2 - d1;
    o3 = d1 - d3;
}

// The 1D output transform A^T applied to four values: (m0 + m1 + m2, m1 - m2 - m3).
__device__ inline void at4(const v4f& m0, const v4f& m1, const v4f& m2, const v4f& m3, v4f& o0,
                           v4f& o1) {
    o0 = m0 + m1 + m2;
    o1 = m1 - m2 - m3;
}

template <int FK, int FT, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void wino_f2x3(WinoArgs a) {
    constexpr int kThreads = WAVES * 64;
    // the transformed filter of the current and of the next channel block:
    // FK output blocks x 16 elements x 64 lane float4 each, double-buffered
    __shared__ v4f ublk[2][FK][kWinoElems][64];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15, g = lane >> 4;
    // logical workgroup: channel tiles fastest, so the workgroups that read
    // one input tile group are neighbours in the XCD's contiguous run
    // (measured on ResNet-50's and VGG-16's 3x3 layers at batch 1 and 32, the
    // other order -- one channel tile's filter slice per XCD, every tile unit
    // -- is within 1 %)
    const int u = __builtin_amdgcn_readfirstlane(xcd_order());
    const int kt = u % a.nkt;
    const int rest = u / a.nkt;
    const int tg = rest % a.ntg;
    const int z = rest / a.ntg;

    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.x), (short)0, a.x_bytes, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t ur =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.u), (short)0, a.u_bytes, kRsrcWord3);

    // the lane's tiles (wave w takes tile groups (tg * WAVES + w) * FT + p):
    // byte offset of every patch position of channel block 0 (the lane's
    // channel quad), or out of range where the position lies in the padding
    unsigned toff[FT][16];
    bool tv[FT];
    int tn[FT], toh[FT], tow[FT];
#pragma unroll
    for (int p = 0; p < FT; ++p) {
        const int tix = ((tg * WAVES + wave) * FT + p) * 16 + li;
        tv[p] = tix < a.NT;  // lanes past the last tile load tile 0 and never store
        const int tt = tv[p] ? tix : 0;
        const int n = fdiv(tt, a.div_tt);
        const int rem = tt - n * a.div_tt.d;
        const int th = fdiv(rem, a.div_tw);
        const int tw = rem - th * a.TW;
        tn[p] = n;
        toh[p] = 2 * th;
        tow[p] = 2 * tw;
        const int ih0 = 2 * th - a.ph, iw0 = 2 * tw - a.pw;
        const int base = ((n * a.CB * a.H + ih0) * a.W + iw0) * 64 + 16 * g;
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const bool ok = (unsigned)(ih0 + i) < (unsigned)a.H && (unsigned)(iw0 + j) < (unsigned)a.W;
                toff[p][4 * i + j] = ok ? (unsigned)(base + (i * a.W + j) * 64) : kOutOfRange;
            }
    }
    // the workgroup's share of one channel block's transformed filter: thread
    // t stages float4s t, t + kThreads, ... of each output block's 16 KB
    constexpr int kPer = kWinoElems * 64 / kThreads;  // float4s per thread and output block
    unsigned ubase[FK];
#pragma unroll
    for (int f = 0; f < FK; ++f)
        ubase[f] = (unsigned)((kt * FK + f) * a.CB * kWinoElems * 1024 + threadIdx.x * 16);

    // this workgroup's channel blocks [k_lo, k_hi)
    const int T = a.CB;
    const int k_lo = __builtin_amdgcn_readfirstlane((int)(((long)T * z) / a.split));
    const int k_hi = __builtin_amdgcn_readfirstlane((int)(((long)T * (z + 1)) / a.split));
    const int dx = __builtin_amdgcn_readfirstlane(a.H * a.W * 64);

    v4f acc[FK][FT][16];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int p = 0; p < FT; ++p)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[f][p][e] = v4f{0.f, 0.f, 0.f, 0.f};

    v4f raw[FT][16];
    v4f ust[FK][kPer];
    auto load_patch = [&](int cb) {
        const int sx = __builtin_amdgcn_readfirstlane(cb * dx);
#pragma unroll
        for (int p = 0; p < FT; ++p)
#pragma unroll
            for (int q = 0; q < 16; ++q) raw[p][q] = ld4(xr, toff[p][q], sx, 0);
    };
    auto load_filter = [&](int cb) {
        const int su = __builtin_amdgcn_readfirstlane(cb * kWinoElems * 1024);
#pragma unroll
        for (int f = 0; f < FK; ++f)
#pragma unroll
            for (int i = 0; i < kPer; ++i) ust[f][i] = ld4(ur, ubase[f], su, i * kThreads * 16);
    };
    auto stage_filter = [&](int buf) {
        v4f* dst = &ublk[buf][0][0][0];
#pragma unroll
        for (int f = 0; f < FK; ++f)
#pragma unroll
            for (int i = 0; i < kPer; ++i) dst[f * kWinoElems * 64 + threadIdx.x + i * kThreads] = ust[f][i];
    };

    if (k_lo < k_hi) {
        load_filter(k_lo);
        load_patch(k_lo);
        stage_filter(0);
        __syncthreads();
        int buf = 0;
        for (int cb = k_lo; cb < k_hi; ++cb) {
            // the next block's filter and patch load while this block's MFMAs
            // run (the last block reloads itself: in range, never used)
            const int nx = cb + 1 < k_hi ? cb + 1 : cb;
            load_filter(nx);
            // B^T d B: the patch's rows combined, then its columns
            v4f V[FT][16];
#pragma unroll
            for (int p = 0; p < FT; ++p) {
                v4f t[4][4];
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    bt4(raw[p][j], raw[p][4 + j], raw[p][8 + j], raw[p][12 + j], t[0][j], t[1][j], t[2][j],
                        t[3][j]);
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    bt4(t[i][0], t[i][1], t[i][2], t[i][3], V[p][4 * i], V[p][4 * i + 1], V[p][4 * i + 2],
                        V[p][4 * i + 3]);
            }
            load_patch(nx);
            // keep the next block's loads here, ahead of the MFMAs: left to
            // itself the scheduler sinks them to their first use at the end of
            // the block, and every block then waits for a full load latency
            __builtin_amdgcn_sched_barrier(0);
            // each element's filter operands are read from LDS one element
            // ahead of its MFMAs, so the read latency hides under the MFMAs
            // of the element before
            v4f uf[2][FK];
#pragma unroll
            for (int f = 0; f < FK; ++f) uf[0][f] = ublk[buf][f][0][lane];
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                if (e + 1 < 16) {
#pragma unroll
                    for (int f = 0; f < FK; ++f) uf[(e + 1) & 1][f] = ublk[buf][f][e + 1][lane];
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int t = 0; t < 4; ++t)
#pragma unroll
                    for (int f = 0; f < FK; ++f)
#pragma unroll
                        for (int p = 0; p < FT; ++p)
                            acc[f][p][e] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                uf[e & 1][f][t], V[p][e][t], acc[f][p][e], 0, 0, 0);
                // fence per element: the next element's reads stay ahead of
                // this element's MFMAs
                __builtin_amdgcn_sched_barrier(0);
            }
            // every wave has read this block's filter once the barrier after
            // the next block's staging passes, so the buffers alternate
            stage_filter(buf ^ 1);
            __syncthreads();
            buf ^= 1;
        }
    }

    // A^T M A: columns combined, then rows; out[..][2 r + c] is output (r, c)
    const int ohw = a.OH * a.OW;
#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kt * FK + f;
        v4f bb = v4f{0.f, 0.f, 0.f, 0.f};
        if (a.split == 1 && a.bias) bb = *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * g);
#pragma unroll
        for (int p = 0; p < FT; ++p) {
            if (!tv[p]) continue;
            const v4f* M = acc[f][p];
            v4f s0[4], s1[4], out[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) at4(M[j], M[4 + j], M[8 + j], M[12 + j], s0[j], s1[j]);
            at4(s0[0], s0[1], s0[2], s0[3], out[0], out[1]);
            at4(s1[0], s1[1], s1[2], s1[3], out[2], out[3]);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int oh = toh[p] + (q >> 1), ow = tow[p] + (q & 1);
                if (oh >= a.OH || ow >= a.OW) continue;  // ragged last tile row / column
                const int pix = oh * a.OW + ow;
                if (a.split > 1) {
                    float* part = a.ws + (long)z * a.N * a.KB * ohw * 16;
                    *reinterpret_cast<v4f*>(part + ((tn[p] * a.KB + kb) * ohw + pix) * 16 + 4 * g) = out[q];
                    continue;
                }
                v4f o = out[q] + bb;
                if (a.res) o += *reinterpret_cast<const v4f*>(a.res + ((tn[p] * a.KB + kb) * ohw + pix) * 16 + 4 * g);
                if (a.act == NEO_ACT_RELU) {
#pragma unroll
                    for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
                }
                *reinterpret_cast<v4f*>(a.y + ((tn[p] * a.y_tot + a.y_off + kb) * ohw + pix) * 16 + 4 * g) = o;
            }
        }
    }
}

// The transformed filter of a KCRS [K][C][3][3] filter (device), zero padded:
// one thread per (output channel, input channel) of the padded blocks.
__global__ __launch_bounds__(256) void wino_filter_kernel(const float* w, int K, int C, float* u) {
    const int CB = (C + 15) / 16, KP = (K + 15) / 16 * 16, CP = CB * 16;
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= KP * CP) return;
    const int k = t / CP, c = t - k * CP;
    float ut[kWinoElems];
    if (k < K && c < C) {
        float g9[9];
        for (int i = 0; i < 9; ++i) g9[i] = w[((long)k * C + c) * 9 + i];
        wino_filter_tile(g9, ut);
    } else {
        for (int e = 0; e < kWinoElems; ++e) ut[e] = 0.f;
    }
    for (int e = 0; e < kWinoElems; ++e) u[wino_filter_index(CB, k, c, e)] = ut[e];
}

template <int FK, int FT, int WAVES>
hipError_t launch_t(const WinoArgs& a, hipStream_t st) {
    const long wgs = (long)a.ntg * a.nkt * a.split;
    hipLaunchKernelGGL((wino_f2x3<FK, FT, WAVES>), dim3((unsigned)wgs), dim3(WAVES * 64), 0, st, a);
    return hipGetLastError();
}

// Eight waves only for the one-tile register tile: two waves per SIMD must
// fit in 256 registers each, which the larger tiles exceed.  The waves share
// the filter stage evenly: 16 float4 per output block over 1 to 8 waves.
template <int FK, int FT>
hipError_t by_waves(int waves, const WinoArgs& a, hipStream_t st) {
    if (waves == 1) return launch_t<FK, FT, 1>(a, st);
    if (waves == 2) return launch_t<FK, FT, 2>(a, st);
    if (waves == 4) return launch_t<FK, FT, 4>(a, st);
    if constexpr (FK * FT == 1) {
        if (waves == 8) return launch_t<FK, FT, 8>(a, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace

bool wino_eligible(const ConvShape& s) {
    return s.R == 3 && s.S == 3 && s.sh == 1 && s.sw == 1 && s.xb == 16 && s.yb == 16 && !s.gap &&
           !conv_small_c(s);
}

bool wino_config_valid(const ConvShape& s, const ConvConfig& c) {
    const int KB = cdiv(s.K, 16), CB = cdiv(s.C, 16);
    // accumulators: 16 * fk * ft float4 per lane (at most 128 registers);
    // the filter stage: 2 * fk * 16 KB of LDS
    const bool tile = ((c.fk == 1 || c.fk == 2) && c.fp == 1) || (c.fk == 1 && c.fp == 2);
    const bool waves = c.waves == 1 || c.waves == 2 || c.waves == 4 || c.waves == 8;
    return wino_eligible(s) && tile && waves && KB % c.fk == 0 && c.split >= 1 && c.split <= CB &&
           c.split <= 64 && (c.waves < 8 || c.fk * c.fp == 1);
}

size_t wino_filter_floats(const ConvShape& s) {
    return (size_t)cdiv(s.K, 16) * cdiv(s.C, 16) * kWinoElems * 256;
}

void wino_filter_host(const float* w, int K, int C, float* u) {
    const int CB = cdiv(C, 16), KP = cdiv(K, 16) * 16, CP = CB * 16;
    for (int k = 0; k < KP; ++k)
        for (int c = 0; c < CP; ++c) {
            float ut[kWinoElems] = {0.f};
            if (k < K && c < C) wino_filter_tile(w + ((long)k * C + c) * 9, ut);
            for (int e = 0; e < kWinoElems; ++e) u[wino_filter_index(CB, k, c, e)] = ut[e];
        }
}

hipError_t launch_wino_filter(const float* w, int K, int C, float* u, hipStream_t st) {
    const long n = (long)cdiv(K, 16) * 16 * cdiv(C, 16) * 16;
    hipLaunchKernelGGL(wino_filter_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, w, K,
                       C, u);
    return hipGetLastError();
}

// Cost model in the spirit of choose_conv_config's: a per-launch floor, plus
// the channel blocks every wave walks (64 * fk * ft MFMAs of 32 cycles each
// per block, shared between the waves resident on a SIMD, and at least the
// ~1.5 us it takes a block's operands to arrive), plus the second kernel and
// partial round trip of a split.
ConvConfig choose_wino_config(const ConvShape& s) {
    const int KB = cdiv(s.K, 16), CB = cdiv(s.C, 16);
    const long NT = (long)s.N * cdiv(s.OH, 2) * cdiv(s.OW, 2);
    const double kClk = 2400.0;
    ConvConfig best{1, 1, 1, 1};
    double best_t = 1e30;
    for (int fk : {1, 2})
        for (int ft : {1, 2})
            for (int wv : {1, 2, 4, 8})
                for (int sp : {1, 2, 4, 8}) {
                    const ConvConfig c{fk, ft, sp, wv};
                    if (!wino_config_valid(s, c)) continue;
                    const long waves = (long)cdiv((int)NT, 16 * ft * wv) * wv * (KB / fk) * sp;
                    const double blocks = std::ceil((double)CB / sp);
                    const double waves_per_simd = (double)waves / 1024.0;
                    const double resident = std::max(1.0, std::min(2.0, waves_per_simd));
                    const double rounds = std::max(1.0, std::ceil(waves_per_simd / 2.0));
                    const double per_block = std::max(64.0 * fk * ft * 32.0 * resident, 1500.0);
                    double t = 3.5 + rounds * blocks * per_block / kClk;
                    if (sp > 1) t += 2.0 + 2.0 * sp * s.N * KB * s.OH * s.OW * 64.0 / 4.0e6;
                    if (t < best_t * 0.98) {
                        best_t = t;
                        best = c;
                    }
                }
    return best;
}

hipError_t launch_wino(const ConvShape& s, const ConvConfig& c, const float* x, const float* u,
                       const float* bias, const float* res, float* y, float* ws, hipStream_t st) {
    if (!wino_config_valid(s, c)) return hipErrorInvalidValue;
    if (c.split > 1 && !ws) return hipErrorInvalidValue;
    WinoArgs a;
    a.x = x;
    a.u = u;
    a.bias = bias;
    a.res = res;
    a.y = y;
    a.ws = ws;
    a.N = s.N;
    a.CB = cdiv(s.C, 16);
    a.H = s.H;
    a.W = s.W;
    a.KB = cdiv(s.K, 16);
    a.OH = s.OH;
    a.OW = s.OW;
    a.ph = s.ph;
    a.pw = s.pw;
    a.TH = cdiv(s.OH, 2);
    a.TW = cdiv(s.OW, 2);
    const long NT = (long)s.N * a.TH * a.TW;
    if (NT >= (1L << 30)) return hipErrorInvalidValue;
    a.NT = (int)NT;
    a.y_off = s.y_off;
    a.y_tot = s.y_tot;
    a.act = s.act;
    a.split = c.split;
    a.ntg = cdiv(a.NT, 16 * c.fp * c.waves);
    a.nkt = a.KB / c.fk;
    a.x_bytes = (int)((long)s.N * a.CB * s.H * s.W * 64);
    a.u_bytes = (int)(wino_filter_floats(s) * 4);
    a.div_tt = make_fastdiv((unsigned)(a.TH * a.TW));
    a.div_tw = make_fastdiv((unsigned)a.TW);
    hipError_t e = hipErrorInvalidValue;
    if (c.fk == 1 && c.fp == 1) e = by_waves<1, 1>(c.waves, a, st);
    if (c.fk == 2 && c.fp == 1) e = by_waves<2, 1>(c.waves, a, st);
    if (c.fk == 1 && c.fp == 2) e = by_waves<1, 2>(c.waves, a, st);
    if (e != hipSuccess || c.split == 1) return e;
    // the direct convolution's second pass: partials added in split order, then the epilogue
    ConvArgs r{};
    r.bias = bias;
    r.res = res;
    r.y = y;
    r.ws = ws;
    r.N = s.N;
    r.KB = a.KB;
    r.OH = s.OH;
    r.OW = s.OW;
    r.y_off = s.y_off;
    r.y_tot = s.y_tot;
    r.act = s.act;
    r.split = c.split;
    return conv_detail::launch_split_reduce(r, st);
}

}  // namespace neo
