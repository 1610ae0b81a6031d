// Blocked convolution on fp32 MFMA (gfx950): the kernel templates.
//
// The convolution of Section 3.1.1 (Algorithm 1) as an implicit GEMM:
//   rows    = output channels k (16 per channel block),
//   columns = output pixels m = (n, oh, ow),
//   reduction over (c, r, s).
// Algorithm 1 keeps reg_n output pixels x y output channels of accumulators in
// vector registers and reduces over (ic.outer, kernel entry, ic.inner).  Here
// the register tile is a set of 16x16 MFMA accumulators: FK channel blocks x
// FP pixel groups per wave, and one reduction step is one (channel block,
// kernel entry) pair = 16 input channels = 4 MFMA k-steps.
//
// v_mfma_f32_16x16x4f32 operand layout (lane l, i = l % 16, g = l / 16):
//   A[i][g] (filter: out channel i, in channel g of the k-step),
//   B[g][i] (input: in channel g, pixel i),
//   D[4g+v][i] in accumulator register v.
// So lane l ends with 4 consecutive output channels (4g..4g+3) of pixel i, and
// the epilogue writes one float4 per lane into the NCHW16c output: 16 pixels x
// 64 bytes = 1 KB contiguous per store instruction.
//
// Input loads: for k-step t the lane needs x[pixel i][channel 4g+t]; one float4
// load at channel offset 4g covers t = 0..3 (the reduction order over the 16
// channels of a block is free).  Filter loads: in the KCRS[16]c[16]k block
// [16 c][16 k] of one (kb, cb, r, s) the lane reads w[c = 4g+t][k = i] (four
// dwords 64 bytes apart); plans store each block as [c/4][k][c%4] instead, so
// the same four values are one float4.
//
// Work split.  Algorithm 1 parallelizes over disjoint output chunks only; at
// batch 1 that leaves too few chunks for 1024 SIMDs, so the reduction is split
// as well:
//   - across the WAVES waves of a workgroup, each owning a contiguous run of
//     steps, summed through LDS in wave order;
//   - optionally across SPLIT workgroups, each owning a contiguous range of
//     steps and writing its raw partial tile to a workspace; a second kernel
//     adds the SPLIT partials in split order (deterministic) and runs the
//     epilogue.  The kernel boundary makes the partials visible across XCDs
//     (whose L2s are not coherent) without a per-workgroup device-scope
//     release, which measured ~20 ns of serialized time per workgroup.  A
//     one-kernel variant (partials stored past the L2, a release, an arrival
//     counter per tile, the last arrival reducing with coherent loads)
//     measured 2-4 % slower end to end at batch 1: its serial chain of store
//     acknowledgement, atomic and loads costs more than the second launch.
// Grouped steps.  A step's bookkeeping (advancing the scalar offsets, the loop
// and ring guards) costs about as many issue cycles as the 4 MFMAs of a one-
// tile step, measured on MI355X.  Small register tiles therefore take G
// channel blocks per step (G = 4 for a 1x1 tile, 2 for a 2-tile one, when G
// divides the channel blocks), so a step issues 4*G*FK*FP MFMAs for one round
// of bookkeeping.
// Loads run D steps ahead of the MFMAs (a register ring of D = 2 slots), so
// each wave keeps D-1 steps of loads in flight while it computes.  The step
// bookkeeping is scalar and incremental (see Loader): measured on MI355X, a
// per-step lane-offset computation, an LDS table or integer divisions per step
// cost more than the MFMAs themselves at batch 1.
// The epilogue (bias, residual, ReLU) runs in registers before the single store.
//
// Small-channel path (C <= 4, the network stems).  A channel block would be
// three quarters padding, and one k-step per kernel entry would need a scalar
// load per lane and entry.  Instead a reduction step is (filter row r, group u
// of 4 filter columns): lane group g takes column s = 4u + g and loads the
// float4 of channels 0..3 of its pixel's input at (r, s), component t feeding
// k-step t.  So the 16 reduction elements of a step are 4 columns x 4
// channels, every operand is one float4 per lane as on the main path, and a
// padding column s >= S reads as 0 like a padding tap.  An NCHW input
// (NCHW1c, block 1) needs no transform: the lane loads its pixel's channels
// one plane apart, and the channels past C read as 0.
#pragma once

#include <algorithm>
#include <cmath>

#include "neo_internal.h"
#include "pool_kernel.h"

namespace neo {
namespace conv_detail {

typedef float v4f __attribute__((ext_vector_type(4)));

// Division by a runtime constant d >= 1 for dividends below 2^31, as a
// multiply-high and a shift (Granlund and Montgomery's round-up method,
// Hacker's Delight 10-9): s = ceil(log2 d), m = floor(2^32 (2^s - d) / d) + 1,
// n / d = (mulhi(n, m) + n) >> s.  The parameters are computed on the host.
struct FastDiv {
    unsigned d, m, s;
};

inline FastDiv make_fastdiv(unsigned d) {
    unsigned s = 0;
    while ((1ull << s) < d) ++s;
    const unsigned long long m = ((1ull << 32) * ((1ull << s) - d)) / d + 1;
    return FastDiv{d, (unsigned)m, s};
}

__device__ inline int fdiv(int n, const FastDiv& f) {
    return (int)((__umulhi((unsigned)n, f.m) + (unsigned)n) >> f.s);
}

struct ConvArgs {
    const float* x;
    const float* w;
    const float* bias;
    const float* res;
    float* y;
    float* ws;  // split partials [SPLIT][N][KB][OH][OW][16]
    int N, CB, CBG, H, W, KB, R, S, RS, U, sh, sw, ph, pw, OH, OW, M, y_off, y_tot, act, T, split;
    // Input NCHW[xb]c: XB blocks per image, xpb bytes per pixel block; the
    // reduction's 16-channel group j starts at byte (j >> lq) * dblk +
    // (j & qm) * 64 of the image (xb >= 16: Q = xb / 16 groups per block).
    int xb, XB, xpb, lq, qm, dblk;
    // Output and residual NCHW[yb]c (lyb = log2 yb): y_off / y_tot in blocks
    // of yb; KBk 16-channel groups are stored (the ones past KB are the zero
    // padding of the last block); the residual has KY blocks.
    int yb, lyb, KBk, KY;
    int x_bytes, w_bytes;
    // 1: global average pooling folded in -- y receives per-16-pixel channel
    // sums [ceil(M / 16)][KB * 16] instead of the outputs (one image, no split)
    int gap;
    FastDiv div_ohw, div_ow, div_npx, div_nkb;
    // 1: logical workgroups take channel tiles first (the workgroups of one
    // pixel tile adjacent, so on one XCD), 0: pixel tiles first
    int kfirst;
};

// Layout arithmetic.  XY = false is the NCHW16c -> NCHW16c kernel, whose
// offsets are compile-time multiples of 64 bytes; XY = true reads the blocks
// from the arguments.
// Byte offset of the reduction's 16-channel group j inside an input image.
__device__ inline int xgroup(const ConvArgs& a, int j) { return (j >> a.lq) * a.dblk + ((j & a.qm) << 6); }
template <bool XY>
__device__ inline int xpb_of(const ConvArgs& a) {
    if constexpr (XY) return a.xpb; else return 64;
}
template <bool XY>
__device__ inline int xblocks(const ConvArgs& a) {
    if constexpr (XY) return a.XB; else return a.CB;
}
// 16-channel output groups stored (the last block's zero padding included)
template <bool XY>
__device__ inline int kgroups(const ConvArgs& a) {
    if constexpr (XY) return a.KBk; else return a.KB;
}
// Float index of channels c..c+3 (c a multiple of 4) of pixel pix = oh * OW +
// ow of image n in an NCHW[yb]c tensor of `tot` blocks per image.
template <bool XY>
__device__ inline int yindex(const ConvArgs& a, int n, int tot, int c, int pix) {
    if constexpr (XY)
        return ((n * tot + (c >> a.lyb)) * (a.OH * a.OW) + pix) * a.yb + (c & (a.yb - 1));
    else
        return ((n * tot + (c >> 4)) * (a.OH * a.OW) + pix) * 16 + (c & 15);
}
template <bool XY>
__device__ inline int rblocks(const ConvArgs& a) {
    if constexpr (XY) return a.KY; else return a.KB;
}

constexpr int kXcds = 8;
constexpr unsigned kRsrcWord3 = 0x00020000;    // raw buffer, gfx9 family
constexpr unsigned kOutOfRange = 0x80000000u;  // buffer offset that reads as 0

template <int FK, int FP, int G>
struct Operands {
    v4f b[G][FP];  // input: lane's pixel, 4 reduction elements (k-steps t = 0..3) per block
    v4f a[G][FK];  // filter: lane's output channel, the same 4 reduction elements
};

// Bits [max(lo, 0), min(hi, n, 32)) set.
__device__ inline unsigned run_mask(int lo, int hi, int n) {
    lo = lo < 0 ? 0 : lo;
    hi = hi > n ? n : hi;
    hi = hi > 32 ? 32 : hi;
    if (hi <= lo) return 0u;
    const unsigned top = hi >= 32 ? 0xffffffffu : ((1u << hi) - 1u);
    return top & ~((1u << lo) - 1u);
}

__device__ inline v4f ld4(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff, int imm) {
    return __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(r, voff + imm, soff, 0));
}
__device__ inline float ld1(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff, int imm) {
    return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, voff + imm, soff, 0));
}

// Per-wave loader.  Reduction steps are taken tap-major, st = rs*CB + cb
// (kernel entry rs = r*S + s outer, channel block cb inner), so within one tap
// the zero-padding test and the per-lane offsets do not change and a step only
// advances two scalar offsets: input += H*W*64 bytes, filter += R*S*1 KB.  The
// per-lane part is recomputed once per tap.  All loads are buffer loads; a
// zero-padding tap gets an out-of-range lane offset, for which the hardware
// returns 0.  Every load is issued unconditionally, so the number of loads in
// flight is static and the compiler waits only for the step it is about to
// use.
//   WMFMA:  filter blocks stored [c/4][k][c%4] (one float4 per lane) instead
//           of the KCRS[16]c[16]k block [c][k] (four dwords, 64 bytes apart).
//   SMALLC: steps st = r*U + u over filter rows and groups of 4 columns; the
//           lane's column s = 4u + g varies by lane group, so the padding
//           test runs every step (it is a few VALU operations).
template <int FK, int FP, int G, bool SMALLC, bool WMFMA, bool XY>
struct Loader {
    __amdgpu_buffer_rsrc_t xr, wr;
    int xoff[FP];                 // byte offset of the lane's pixel at (group, r, s) = 0 (may be < 0)
    unsigned rowm[FP], colm[FP];  // bit r / s set when that tap row / column is inside
    int pih[FP], piw[FP];
    unsigned woff[FK];            // byte offset of the lane's element in filter block (kb, 0, 0)
    bool wide_taps;               // more than 32 taps per axis: explicit test
    int lg;                       // lane group g (small-channel column offset)
    // position of the next step to load (wave-uniform)
    int st, cb, rs, r, s;         // small-channel path: s holds the column group u
    int sx, sw;                   // step byte offsets: input group cb, filter (cb*RS + rs)*1024
    int dx, dw;                   // one channel group further: input H*W*64 (XY = false), filter RS*1024
    int ioff[G];                  // XY: input offset of group cb + i from group cb (cb % G == 0)
    unsigned toff[FP];            // lane offset of the current tap, or out of range
    unsigned wtoff[FK];           // small-channel, KCRS[16]c[16]k filter: lane offset or out of range
    int plain_c, plane;           // small-channel NCHW input: its channels (0 otherwise), bytes per channel

    __device__ void set_tap(const ConvArgs& a) {
        if constexpr (SMALLC) {
            const int sc = 4 * s + lg;
            const bool cok = sc < a.S;
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                bool ok;
                if (!wide_taps)
                    ok = cok && (((rowm[p] >> r) & (colm[p] >> sc) & 1u) != 0);
                else
                    ok = cok && (unsigned)(pih[p] + r) < (unsigned)a.H &&
                         (unsigned)(piw[p] + sc) < (unsigned)a.W;
                toff[p] = ok ? (unsigned)(xoff[p] + (r * a.W + sc) * xpb_of<XY>(a)) : kOutOfRange;
            }
            if constexpr (!WMFMA) {
#pragma unroll
                for (int f = 0; f < FK; ++f) wtoff[f] = cok ? woff[f] : kOutOfRange;
            }
        } else {
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                bool ok;
                if (!wide_taps)
                    ok = ((rowm[p] >> r) & (colm[p] >> s) & 1u) != 0;
                else
                    ok = (unsigned)(pih[p] + r) < (unsigned)a.H && (unsigned)(piw[p] + s) < (unsigned)a.W;
                toff[p] = ok ? (unsigned)(xoff[p] + (r * a.W + s) * xpb_of<XY>(a)) : kOutOfRange;
            }
        }
    }
    // The step state is wave-uniform; readfirstlane pins it to scalar
    // registers (otherwise the compiler may keep it in vector registers and
    // wrap every buffer load, whose soffset must be scalar, in a waterfall
    // loop).
    __device__ void pin() {
        st = __builtin_amdgcn_readfirstlane(st);
        cb = __builtin_amdgcn_readfirstlane(cb);
        rs = __builtin_amdgcn_readfirstlane(rs);
        r = __builtin_amdgcn_readfirstlane(r);
        s = __builtin_amdgcn_readfirstlane(s);
        sx = __builtin_amdgcn_readfirstlane(sx);
        sw = __builtin_amdgcn_readfirstlane(sw);
    }
    // filter step offset of the small-channel path at (r, u)
    __device__ int small_sw(const ConvArgs& a) const {
        return WMFMA ? (r * a.U + s) * 1024 : (r * a.S + 4 * s) * 1024;
    }
    __device__ void seek(const ConvArgs& a, int st0) {
        st = st0;
        if constexpr (SMALLC) {
            r = st0 / a.U;
            s = st0 - r * a.U;
            cb = 0;
            rs = 0;
            sx = 0;
            sw = small_sw(a);
        } else {
            rs = st0 / a.CBG;
            cb = (st0 - rs * a.CBG) * G;
            r = rs / a.S;
            s = rs - r * a.S;
            sx = XY ? xgroup(a, cb) : cb * a.H * a.W * 64;
            sw = (cb * a.RS + rs) * 1024;
        }
        dx = __builtin_amdgcn_readfirstlane(a.H * a.W * 64);
        dw = __builtin_amdgcn_readfirstlane(a.RS * 1024);
        if constexpr (XY) {
            // cb stays a multiple of G and G, Q are powers of two, so group
            // cb + i (i < G) lies xgroup(i) bytes past group cb
#pragma unroll
            for (int i = 0; i < G; ++i) ioff[i] = __builtin_amdgcn_readfirstlane(xgroup(a, i));
        }
        pin();
        set_tap(a);
    }
    __device__ void next(const ConvArgs& a) {
        ++st;
        if constexpr (SMALLC) {
            if (++s == a.U) {
                s = 0;
                ++r;
            }
            sw = small_sw(a);
            pin();
            set_tap(a);
        } else if ((cb += G) < a.CB) {
            if constexpr (XY)
                sx = xgroup(a, cb);
            else
                sx += G * dx;
            sw += G * dw;
        } else {
            cb = 0;
            ++rs;
            sx = 0;
            sw = rs * 1024;
            if (++s == a.S) {
                s = 0;
                ++r;
            }
            pin();
            set_tap(a);
        }
        pin();
    }
    __device__ void load(Operands<FK, FP, G>& o) const {
#pragma unroll
        for (int i = 0; i < G; ++i) {
            const int sxi = sx + (XY ? ioff[i] : i * dx), swi = sw + i * dw;
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                if constexpr (SMALLC && XY) {
                    if (plain_c) {  // NCHW: the pixel's channels lie a plane apart; the rest are 0
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            o.b[i][p][t] = t < plain_c ? ld1(xr, toff[p], sxi + t * plane, 0) : 0.f;
                        continue;
                    }
                }
                o.b[i][p] = ld4(xr, toff[p], sxi, 0);
            }
#pragma unroll
            for (int f = 0; f < FK; ++f) {
                if constexpr (WMFMA) {
                    o.a[i][f] = ld4(wr, woff[f], swi, 0);
                } else {
                    const unsigned off = SMALLC ? wtoff[f] : woff[f];
#pragma unroll
                    for (int t = 0; t < 4; ++t) o.a[i][f][t] = ld1(wr, off, swi, t * 64);
                }
            }
        }
    }
};

// Depth of the load ring: two slots, i.e. the next step's operands load
// while this step's MFMAs run.  Measured on MI355X over every ResNet-50
// layer, tuned: sizing the ring to ~72 VGPRs (3 to 8 slots) was 7 % slower
// end to end at batch 1 and 32, twice that budget slower still; the fewer
// registers a wave holds, the more waves share each SIMD and hide latency.
template <int FK, int FP, int G>
constexpr int pipe_depth() {
    return 2;
}

template <int FK, int FP, int G>
__device__ inline void mma(const Operands<FK, FP, G>& o, v4f (&acc)[FK][FP]) {
#pragma unroll
    for (int i = 0; i < G; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[i][f][t], o.b[i][p][t],
                                                                     acc[f][p], 0, 0, 0);
}

// Workgroups are dispatched round-robin over the 8 XCDs, each with its own L2.
// The logical workgroup index gives every XCD a contiguous run of the logical
// order (member, split, channel tile, pixel tile), so the pixel tiles that
// share a filter slice run on one XCD and read it from that XCD's L2.
// (For workgroup b of the first nwg of the grid.)
__device__ inline int xcd_order(int b, int nwg) {
    const int xcd = b % kXcds, slot = b / kXcds;
    const int q = nwg / kXcds, rmd = nwg % kXcds;
    return xcd * q + min(xcd, rmd) + slot;
}
__device__ inline int xcd_order() { return xcd_order(blockIdx.x, gridDim.x); }

// One workgroup's output tile: logical workgroup u of the convolution a.
template <int FK, int FP, int G, bool SMALLC, bool WMFMA, int WAVES, bool XY>
__device__ __forceinline__ void conv_tile(const ConvArgs& a, const int u) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15;
    const int g = lane >> 4;
    const int npx = a.div_npx.d, nkb = a.div_nkb.d;
    int pxt, kbt, z;
    if (a.kfirst) {
        const int u_k = fdiv(u, a.div_nkb);
        kbt = u - u_k * nkb;
        z = fdiv(u_k, a.div_npx);
        pxt = u_k - z * npx;
    } else {
        const int u_px = fdiv(u, a.div_npx);
        pxt = u - u_px * npx;
        z = fdiv(u_px, a.div_nkb);
        kbt = u_px - z * nkb;
    }
    const int m0 = pxt * (16 * FP);
    const int kb0 = kbt * FK;
    const int ohw = a.OH * a.OW;

    Loader<FK, FP, G, SMALLC, WMFMA, XY> tl;
    tl.xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.x), (short)0, a.x_bytes, kRsrcWord3);
    tl.wr = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.w), (short)0, a.w_bytes, kRsrcWord3);
    tl.wide_taps = a.R > 32 || a.S > 32;
    tl.lg = g;
    tl.plain_c = __builtin_amdgcn_readfirstlane(XY && a.xb == 1 ? (a.XB < 4 ? a.XB : 4) : 0);
    tl.plane = __builtin_amdgcn_readfirstlane(a.H * a.W * 4);
    bool pv[FP];
    int pn[FP];
#pragma unroll
    for (int p = 0; p < FP; ++p) {
        const int m = m0 + 16 * p + li;
        pv[p] = m < a.M;  // lanes past the last pixel load pixel 0 and never store
        const int mm = pv[p] ? m : 0;
        const int n = fdiv(mm, a.div_ohw);
        const int rem = mm - n * ohw;
        const int oh = fdiv(rem, a.div_ow);
        pn[p] = n;
        const int ih0 = oh * a.sh - a.ph;
        const int iw0 = (rem - oh * a.OW) * a.sw - a.pw;
        tl.pih[p] = ih0;
        tl.piw[p] = iw0;
        // taps r with 0 <= ih0 + r < H form the run [-ih0, H - ih0) of [0, R)
        tl.rowm[p] = run_mask(-ih0, a.H - ih0, a.R);
        tl.colm[p] = run_mask(-iw0, a.W - iw0, a.S);
        // byte offset of this pixel's (group 0, r = 0, s = 0) element, the lane's
        // channel quad 4g..4g+3 of the group; only used (with a step offset
        // added) when the tap is inside the input
        tl.xoff[p] = ((n * xblocks<XY>(a) * a.H + ih0) * a.W + iw0) * xpb_of<XY>(a) + (SMALLC ? 0 : 16 * g);
    }
#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kb0 + f < a.KB ? kb0 + f : 0;  // past K: clamped, result stored as zero
        if constexpr (SMALLC) {
            // kernel order: block (kb, r, u), lane's float4 at (g*16 + k)*4;
            // KCRS[16]c[16]k: block (kb, r, s = 4u + g), element [c][k]
            tl.woff[f] = WMFMA ? (unsigned)((kb * a.R * a.U * 256 + (g * 16 + li) * 4) * 4)
                               : (unsigned)((kb * a.RS * 256 + g * 256 + li) * 4);
        } else {
            const int e = WMFMA ? (g * 16 + li) * 4 : (4 * g) * 16 + li;
            tl.woff[f] = (unsigned)((kb * a.CB * a.RS * 256 + e) * 4);
        }
    }

    v4f acc[FK][FP];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int p = 0; p < FP; ++p) acc[f][p] = v4f{0.f, 0.f, 0.f, 0.f};

    // The epilogue's bias and residual reads are issued now, by the wave that
    // runs the epilogue, so their latency hides under the reduction -- for
    // small register tiles only: the FK * FP held residuals cost registers,
    // and so waves per SIMD, which larger tiles need more (measured: holding
    // them for tiles of up to 8 was 2.5 % slower at batch 32, equal at batch 1).
    constexpr bool kPrefetch = FK * FP <= (WAVES >= 4 ? 4 : 2);
    v4f pre_b[kPrefetch ? FK : 1], pre_r[kPrefetch ? FK : 1][kPrefetch ? FP : 1];
    if constexpr (kPrefetch) {
        if (wave == 0 && a.split == 1) {
#pragma unroll
            for (int f = 0; f < FK; ++f) {
                const int kb = kb0 + f < a.KB ? kb0 + f : 0;
                pre_b[f] = a.bias ? *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * g)
                                  : v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int p = 0; p < FP; ++p) {
                    const int oh = (tl.pih[p] + a.ph) / a.sh;
                    const int ow = (tl.piw[p] + a.pw) / a.sw;
                    pre_r[f][p] = a.res ? *reinterpret_cast<const v4f*>(
                                              a.res + yindex<XY>(a, pn[p], rblocks<XY>(a), kb * 16 + 4 * g, oh * a.OW + ow))
                                        : v4f{0.f, 0.f, 0.f, 0.f};
                }
            }
        }
    }

    // this workgroup's contiguous range of reduction steps, cut into one
    // contiguous run per wave
    const int k_lo = (int)(((long)a.T * z) / a.split);
    const int k_hi = (int)(((long)a.T * (z + 1)) / a.split);
    const int w_lo = k_lo + (int)(((long)(k_hi - k_lo) * wave) / WAVES);
    const int w_hi = k_lo + (int)(((long)(k_hi - k_lo) * (wave + 1)) / WAVES);
    const int nj = w_hi - w_lo;

    if (nj > 0) {
        constexpr int D = pipe_depth<FK, FP, G>();
        // the loader runs D - 1 steps ahead; past the wave's last step it
        // stays there (those loads are never consumed)
        tl.seek(a, w_lo);
        Operands<FK, FP, G> buf[D];
#pragma unroll
        for (int i = 0; i < D - 1; ++i) {
            tl.load(buf[i]);
            if (tl.st < w_hi - 1) tl.next(a);
        }
        // Steady state: while two more rings of steps remain, the loader never
        // reaches the wave's last step and every slot is consumed, so the
        // ring runs without guards.  At block j0 the loader stands at step
        // j0 + D - 1 and loads up to j0 + 2D - 2 < nj - 1.
        int j0 = 0;
        for (; j0 + 2 * D <= nj; j0 += D) {
#pragma unroll
            for (int uu = 0; uu < D; ++uu) {
                // refill the slot consumed one step ago with step j0 + uu + D - 1
                tl.load(buf[(uu + D - 1) % D]);
                tl.next(a);
                mma<FK, FP, G>(buf[uu], acc);
            }
        }
        for (; j0 < nj; j0 += D) {
#pragma unroll
            for (int uu = 0; uu < D; ++uu) {
                const int j = j0 + uu;
                tl.load(buf[(uu + D - 1) % D]);
                if (tl.st < w_hi - 1) tl.next(a);
                if (j < nj) mma<FK, FP, G>(buf[uu], acc);
            }
        }
    }

    // Sum the waves' partial tiles in wave order: 0 + 1 + 2 + ...
    if constexpr (WAVES > 1) {
        __shared__ v4f red[WAVES - 1][FK * FP][64];
        if (wave > 0) {
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p) red[wave - 1][f * FP + p][lane] = acc[f][p];
        }
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int f = 0; f < FK; ++f)
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                const int qq = f * FP + p;
#pragma unroll
                for (int w = 0; w < WAVES - 1; ++w) acc[f][p] += red[w][qq][lane];
            }
    }

    if (a.split > 1) {
        // raw partial sums of split z, in the output's own blocked layout; the
        // reduce kernel adds the splits in order and runs the epilogue
        float* part = a.ws + (long)z * a.N * a.KB * ohw * 16;
#pragma unroll
        for (int f = 0; f < FK; ++f) {
            const int kb = kb0 + f;
            if (kb >= a.KB) continue;
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                if (!pv[p]) continue;
                const int oh = (tl.pih[p] + a.ph) / a.sh;
                const int ow = (tl.piw[p] + a.pw) / a.sw;
                *reinterpret_cast<v4f*>(part + (((pn[p] * a.KB + kb) * a.OH + oh) * a.OW + ow) * 16 +
                                        4 * g) = acc[f][p];
            }
        }
        return;
    }

    // act(acc + bias + residual) of pixel group p, channel quad of output group kb
    auto out_value = [&](const v4f& sum, const v4f& bb, const v4f& pre, int p, int kb) {
        v4f o = sum + bb;
        if constexpr (kPrefetch) {
            o += pre;
        } else if (a.res) {
            const int oh = (tl.pih[p] + a.ph) / a.sh;
            const int ow = (tl.piw[p] + a.pw) / a.sw;
            o += *reinterpret_cast<const v4f*>(
                a.res + yindex<XY>(a, pn[p], rblocks<XY>(a), kb * 16 + 4 * g, oh * a.OW + ow));
        }
        if (a.act == NEO_ACT_RELU) {
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
        }
        return o;
    };

#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kb0 + f;
        if (kb >= kgroups<XY>(a)) continue;
        // groups past the last real one only fill the last output block with zeros
        const bool real = kb < a.KB;
        v4f bb = v4f{0.f, 0.f, 0.f, 0.f};
        if constexpr (kPrefetch)
            bb = pre_b[f];
        else if (a.bias && real)
            bb = *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * g);
#pragma unroll
        for (int p = 0; p < FP; ++p) {
            const v4f pre = pre_r[kPrefetch ? f : 0][kPrefetch ? p : 0];
            if (a.gap) {
                // Global average pooling folded in (one image): instead of the
                // outputs, the sum of this group's 16 pixels per channel, row
                // m / 16 of a [pixel group][KB * 16] table, summed over the 16
                // lanes that hold them in a fixed order.
                const int m = m0 + 16 * p;
                if (!real || m >= a.M) continue;  // the whole wave
                v4f o = pv[p] ? out_value(acc[f][p], bb, pre, p, kb) : v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int off = 8; off > 0; off >>= 1)
#pragma unroll
                    for (int v = 0; v < 4; ++v) o[v] += __shfl_xor(o[v], off, 16);
                if (li == 0) *reinterpret_cast<v4f*>(a.y + (long)(m >> 4) * a.KB * 16 + kb * 16 + 4 * g) = o;
                continue;
            }
            if (!pv[p]) continue;
            const int oh = (tl.pih[p] + a.ph) / a.sh;
            const int ow = (tl.piw[p] + a.pw) / a.sw;
            const v4f o = real ? out_value(acc[f][p], bb, pre, p, kb) : v4f{0.f, 0.f, 0.f, 0.f};
            *reinterpret_cast<v4f*>(
                a.y + yindex<XY>(a, pn[p], a.y_tot, a.y_off * (XY ? a.yb : 16) + kb * 16 + 4 * g, oh * a.OW + ow)) = o;
        }
    }
}

template <int FK, int FP, int G, bool SMALLC, bool WMFMA, int WAVES, bool XY>
__global__ __launch_bounds__(WAVES * 64) void conv2d_mfma(ConvArgs a) {
    conv_tile<FK, FP, G, SMALLC, WMFMA, WAVES, XY>(a, xcd_order());
}

// Several independent convolutions in one launch (horizontal fusion, for
// batch 1 where each is too small to fill the chip and a launch costs more
// than its work).  Member m owns the workgroups [start[m], start[m+1]) of
// the grid, cnt[m] of them real; every start is a multiple of the XCD count,
// so workgroup start[m] + b runs on XCD b % kXcds and each member is spread
// over all XCDs (a member's tiles on a few XCDs would share their CUs while
// the rest idle), its tiles in the same per-XCD order as a launch of its own.
// The last start[m+1] - start[m] - cnt[m] (< kXcds) workgroups of a member
// exit at once.  Every member uses the same kernel parameters and no split
// reduction.
// A pooling step may ride along in workgroups past the convs' (wgs of them,
// grid-stride over its output quads, the same arithmetic as the pooling
// kernel); it is independent of the convs.  Those workgroups come last in
// dispatch order, which spreads them over the XCDs.
constexpr int kMaxGroup = 4;
struct PoolPart {
    const float* x;
    float* y;
    PoolShape s;
    int CB, lq, total, max, k33, wgs;  // wgs = 0: no pooling step
    PoolQ q;                           // its int8 copy (integer group launches only)
};
struct ConvGroupArgs {
    ConvArgs a[kMaxGroup];
    int start[kMaxGroup + 1];
    int cnt[kMaxGroup];
    int n;
    PoolPart pool;
};

template <bool MAX, int K, bool Q = false>
__device__ inline void pool_part_run(const PoolPart& p, int wg) {
    for (int t = wg * blockDim.x + threadIdx.x; t < p.total; t += p.wgs * blockDim.x)
        pool_detail::pool_elem<MAX, K, K, Q>(p.x, p.y, p.s, p.CB, p.lq, t, p.q);
}

template <int FK, int FP, int G, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void conv2d_mfma_group(ConvGroupArgs ga) {
    const int nconv = ga.start[ga.n];
    if ((int)blockIdx.x >= nconv) {
        const int wg = blockIdx.x - nconv;
        if (ga.pool.max)
            ga.pool.k33 ? pool_part_run<true, 3>(ga.pool, wg) : pool_part_run<true, 0>(ga.pool, wg);
        else
            ga.pool.k33 ? pool_part_run<false, 3>(ga.pool, wg) : pool_part_run<false, 0>(ga.pool, wg);
        return;
    }
    int m = 0;
    while (m + 1 < ga.n && (int)blockIdx.x >= ga.start[m + 1]) ++m;
    m = __builtin_amdgcn_readfirstlane(m);
    const int b = blockIdx.x - ga.start[m];
    if (b >= ga.cnt[m]) return;
    conv_tile<FK, FP, G, false, true, WAVES, false>(ga.a[m], xcd_order(b, ga.cnt[m]));
}

// Second pass of a split reduction: y = act(sum_z part[z] + bias + res), the
// splits added in order z = 0, 1, ... (deterministic).  One thread per
// (pixel, 4-channel quad).
template <bool XY>
__global__ __launch_bounds__(256) void split_reduce(ConvArgs a) {
    const int ohw = a.OH * a.OW;
    const int KBk = kgroups<XY>(a);
    const int total = a.N * KBk * ohw * 4;
    const long zstride = (long)a.N * a.KB * ohw * 16;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int qd = t & 3;
        const int pix = t >> 2;  // (n*KBk + kb)*OH*OW + oh*OW + ow
        const int sp = pix % ohw;
        const int nk = pix / ohw;
        const int kb = nk % KBk, n = nk / KBk;
        v4f o = v4f{0.f, 0.f, 0.f, 0.f};
        if (kb < a.KB) {  // past KB: the zero padding of the last output block
            const int part = ((n * a.KB + kb) * ohw + sp) * 16 + 4 * qd;
            o = *reinterpret_cast<const v4f*>(a.ws + part);
            for (int z = 1; z < a.split; ++z)
                o += *reinterpret_cast<const v4f*>(a.ws + z * zstride + part);
            if (a.bias) o += *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * qd);
            if (a.res) o += *reinterpret_cast<const v4f*>(a.res + yindex<XY>(a, n, rblocks<XY>(a), kb * 16 + 4 * qd, sp));
            if (a.act == NEO_ACT_RELU) {
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
            }
        }
        *reinterpret_cast<v4f*>(a.y + yindex<XY>(a, n, a.y_tot, a.y_off * (XY ? a.yb : 16) + kb * 16 + 4 * qd, sp)) = o;
    }
}

// The second pass alone, NCHW16c -> NCHW16c (also for the Winograd kernel,
// whose split partials are raw outputs in the same layout).  Reads a.N, KB,
// OH, OW, ws, split, bias, res, act, y, y_off, y_tot.
inline hipError_t launch_split_reduce(const ConvArgs& a, hipStream_t st) {
    const long total = (long)a.N * a.KB * a.OH * a.OW * 4;
    long blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(split_reduce<false>, dim3((unsigned)blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

template <int FK, int FP, int G, bool SMALLC, bool WMFMA, int WAVES, bool XY>
hipError_t launch_t(const ConvArgs& a, hipStream_t st) {
    const int wgs = cdiv(a.M, 16 * FP) * cdiv(a.KBk, FK) * a.split;
    hipLaunchKernelGGL((conv2d_mfma<FK, FP, G, SMALLC, WMFMA, WAVES, XY>), dim3(wgs),
                       dim3(WAVES * 64), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.split == 1) return e;
    const long total = (long)a.N * a.KBk * a.OH * a.OW * 4;
    long blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(split_reduce<XY>, dim3((unsigned)blocks), dim3(256), 0, st, a);
    return hipGetLastError();
}

// LDS for the cross-wave sum is (WAVES - 1) * FK * FP KB; the instantiated
// combinations keep it at or below 48 KB.  One or two waves per workgroup
// suit short reductions (a 1x1 layer over few channels), where splitting the
// reduction across more waves buys nothing but the LDS sum.
template <int FK, int FP, int G, bool SMALLC, bool WMFMA, bool XY>
hipError_t by_waves(int waves, const ConvArgs& a, hipStream_t st) {
    if (waves == 1) return launch_t<FK, FP, G, SMALLC, WMFMA, 1, XY>(a, st);
    if (waves == 2) return launch_t<FK, FP, G, SMALLC, WMFMA, 2, XY>(a, st);
    if constexpr (FK * FP <= 2) {
        if (waves == 16) return launch_t<FK, FP, G, SMALLC, WMFMA, 16, XY>(a, st);
    }
    if constexpr (FK * FP <= 4) {
        if (waves == 8) return launch_t<FK, FP, G, SMALLC, WMFMA, 8, XY>(a, st);
    }
    if (waves == 4) return launch_t<FK, FP, G, SMALLC, WMFMA, 4, XY>(a, st);
    return hipErrorInvalidValue;
}

// Channel blocks per step: instantiated for G up to 4 / (FK * FP) (1 on the
// small-channel path, whose step is not a channel block).
template <int FK, int FP, bool SMALLC, bool WMFMA, bool XY>
hipError_t by_group(int g, int waves, const ConvArgs& a, hipStream_t st) {
    if constexpr (!SMALLC && FK * FP == 1) {
        if (g == 4) return by_waves<FK, FP, 4, SMALLC, WMFMA, XY>(waves, a, st);
    }
    if constexpr (!SMALLC && FK * FP <= 2) {
        if (g == 2) return by_waves<FK, FP, 2, SMALLC, WMFMA, XY>(waves, a, st);
    }
    if (g == 1) return by_waves<FK, FP, 1, SMALLC, WMFMA, XY>(waves, a, st);
    return hipErrorInvalidValue;
}

template <bool SMALLC, bool WMFMA, bool XY>
hipError_t dispatch(const ConvConfig& c, int g, const ConvArgs& a, hipStream_t st) {
    switch (c.fk * 8 + c.fp) {
        case 1 * 8 + 1: return by_group<1, 1, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 1 * 8 + 2: return by_group<1, 2, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 1 * 8 + 4: return by_group<1, 4, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 2 * 8 + 1: return by_group<2, 1, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 2 * 8 + 2: return by_group<2, 2, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 2 * 8 + 4: return by_group<2, 4, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 4 * 8 + 1: return by_group<4, 1, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 4 * 8 + 2: return by_group<4, 2, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        case 4 * 8 + 4: return by_group<4, 4, SMALLC, WMFMA, XY>(g, c.waves, a, st);
        default: return hipErrorInvalidValue;
    }
}


// Group launches: the NCHW16c family only, no split (conv_group.hip).
template <int FK, int FP, int G, int WAVES>
hipError_t launch_group_t(const ConvGroupArgs& ga, int wgs, hipStream_t st) {
    hipLaunchKernelGGL((conv2d_mfma_group<FK, FP, G, WAVES>), dim3(wgs), dim3(WAVES * 64), 0, st, ga);
    return hipGetLastError();
}

template <int FK, int FP, int G>
hipError_t group_by_waves(int waves, const ConvGroupArgs& ga, int wgs, hipStream_t st) {
    if (waves == 1) return launch_group_t<FK, FP, G, 1>(ga, wgs, st);
    if (waves == 2) return launch_group_t<FK, FP, G, 2>(ga, wgs, st);
    if (waves == 4) return launch_group_t<FK, FP, G, 4>(ga, wgs, st);
    if constexpr (FK * FP <= 4) {
        if (waves == 8) return launch_group_t<FK, FP, G, 8>(ga, wgs, st);
    }
    if constexpr (FK * FP <= 2) {
        if (waves == 16) return launch_group_t<FK, FP, G, 16>(ga, wgs, st);
    }
    return hipErrorInvalidValue;
}

template <int FK, int FP>
hipError_t group_by_g(int g, int waves, const ConvGroupArgs& ga, int wgs, hipStream_t st) {
    if constexpr (FK * FP == 1) {
        if (g == 4) return group_by_waves<FK, FP, 4>(waves, ga, wgs, st);
    }
    if constexpr (FK * FP <= 2) {
        if (g == 2) return group_by_waves<FK, FP, 2>(waves, ga, wgs, st);
    }
    if (g == 1) return group_by_waves<FK, FP, 1>(waves, ga, wgs, st);
    return hipErrorInvalidValue;
}

// Defined in conv_group.hip.
hipError_t dispatch_group(const ConvConfig& c, int g, const ConvGroupArgs& ga, int wgs,
                          hipStream_t st);

// Every launch configuration and path of one kernel family: XY = false for
// NCHW16c in and out, XY = true for any other pair of blocks.  Instantiated
// in conv.hip (false) and conv_xy.hip (true), so the two compile in parallel.
template <bool XY>
hipError_t dispatch_all(const ConvConfig& c, int g, bool small, bool wmfma, const ConvArgs& a,
                        hipStream_t st) {
    if (wmfma) return small ? dispatch<true, true, XY>(c, g, a, st) : dispatch<false, true, XY>(c, g, a, st);
    return small ? dispatch<true, false, XY>(c, g, a, st) : dispatch<false, false, XY>(c, g, a, st);
}

}  // namespace conv_detail
}  // namespace neo
