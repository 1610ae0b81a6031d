// Integer (INT8) convolution on MFMA (gfx950) -- the paper's other future
// work beside fast convolution algorithms (Sections 1 and 5): symmetric linear
// quantization with exact integer accumulation.
//
//   - Activations are int8 in the blocked layout, NCHW16c (16 bytes per
//     pixel block), stored with the convolution's zero padding as an explicit
//     halo: [N][CB][H + 2 ph][W + 2 pw][16].  The quantization pass writes the
//     halo, so every tap of every output pixel is an in-bounds read and the
//     reduction loop has no bounds tests.  A reduction step is one kernel
//     entry (r, s) and one group of 64 input channels (four 16-channel
//     blocks): lane (i, g) loads the 16 bytes of block 4 cg + g of its pixel i
//     with one buffer load; a lane whose block does not exist (C not a
//     multiple of 64) loads from an out-of-range offset, which reads 0
//     without memory traffic.
//   - v_mfma_i32_16x16x64_i8 takes 16 int8 per lane for A (filter, output
//     channel i) and B (input, pixel i); lane group g and byte b of both name
//     the same input channel 64 cg + 16 g + b, so the instruction sums over
//     all 64 whatever its internal order.  Filters are packed so that the A
//     operand is one 16-byte load too, in step order: block (kb, r, s, cg)
//     holds, for lane (k, g), w[16 kb + k][64 cg + 16 g + b][r][s], b = 0..15.
//   - A wave's instruction stream, not the matrix unit, bounds this kernel at
//     the one or two waves per SIMD these layers give (a single wave issues
//     about one instruction per eight cycles; one MFMA here is sixteen): the
//     step decode is scalar and incremental, the loop issues per step only the
//     loads, one address add per input load and the MFMAs, and the epilogue
//     addresses are precomputed per pixel.
//   - The int32 accumulator is exact (|sum| <= 127^2 * C * R * S), and the
//     waves of a workgroup add their partial tiles through LDS (integer sums:
//     any order gives the same bits).  The MFMA result layout is the fp32
//     kernel's: lane (i, g) holds output channels 4 g .. 4 g + 3 of pixel i.
//   - Epilogue: y = act(acc * (s_x * s_w[k]) + bias[k] + residual) in float32,
//     one float4 store into the NCHW16c output view; or (the _acc entry point)
//     the raw int32 accumulators.
#include <algorithm>
#include <cstdint>

#include "conv_kernel.h"

namespace neo {

using conv_detail::FastDiv;
using conv_detail::fdiv;
using conv_detail::kOutOfRange;
using conv_detail::kRsrcWord3;
using conv_detail::make_fastdiv;
using conv_detail::v4f;
using conv_detail::xcd_order;

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kQMax = 127;

struct I8Args {
    const int8_t* x;      // int8 NCHW16c with halo [N][CB][Hp][Wp][16]
    const int8_t* w;      // packed [KB][R][S][CG][64 lanes][16 bytes]
    const float* wscale;  // [KB * 16] per-output-channel filter scales
    float xscale;         // the activations' scale
    const float* bias;    // [KB * 16] or null
    const float* res;     // fp32 NCHW16c [N][KB][OH][OW][16] or null
    float* y;             // fp32 NCHW16c view: blocks [y_off, y_off + KB) of y_tot
    int* acc;             // raw mode: int32 NCHW16c [N][KB][OH][OW][16]
    int8_t* yq;           // int8 modes: NCHW16c with a halo [N][KB][OH + 2 qph][OW + 2 qpw][16]
    float yrcp;           // int8 mode: 1 / (the output's scale), rounded to float32
    float ydiv;           // > 0: requantize by division by this scale instead
    int qph, qpw;         // int8 modes: the output's halo
    int q_off, q_tot;     // int8 modes: blocks [q_off, q_off + KB) of q_tot
    int N, CB, CG, Hp, Wp, KB, S, sh, sw, OH, OW, M, y_off, y_tot, act;
    int hoff, woff;       // x's halo beyond the conv's padding (rows, columns)
    int T;                // reduction steps: R * S * CG
    int npx, nkt;         // pixel tiles (16 * FP pixels), channel tiles (FK blocks)
    int ntiles;           // npx * nkt
    int x_bytes, w_bytes;
    FastDiv div_ohw, div_ow, div_npx;
};

__device__ inline v4i ld16(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
    return __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// A wave's position in its run of reduction steps st = (r * S + s) * CG + cg:
// the step, its channel group and kernel column, and the input bytes the
// channel group and tap add to a window's first byte.
struct StepCursor {
    int st, cg, s, uoff;
};
// The run's constants: the last step and the uoff increments to the next
// channel group, the next tap of a kernel row and the next kernel row.
struct StepGeometry {
    int CG, S, hi, d_cg, d_s, d_r;
};

// Issue the loads of the cursor's step (input pixel blocks, filter blocks)
// and advance the cursor, unless it is at the run's last step.
template <int FK, int FP>
__device__ __forceinline__ void load_step(const __amdgpu_buffer_rsrc_t xr, const __amdgpu_buffer_rsrc_t wr,
                                          const int (&xbase)[FP], const unsigned (&woff)[FK], const int glim,
                                          const StepGeometry geo, StepCursor& c, v4i (&A)[FK], v4i (&B)[FP]) {
    // a lane whose channel block 4 cg + g does not exist (C <= 48, or the last
    // group of a C that is not a multiple of 64) reads nothing: its filter
    // bytes are zero, and the out-of-range offset costs no memory traffic
    const bool gok = 4 * c.cg < glim;
#pragma unroll
    for (int p = 0; p < FP; ++p) B[p] = ld16(xr, gok ? (unsigned)(xbase[p] + c.uoff) : kOutOfRange, 0);
#pragma unroll
    for (int f = 0; f < FK; ++f) A[f] = ld16(wr, woff[f], c.st * 1024);
    // scalar selects, not a branch tree: the compiler turned the branches
    // into a load of the increment from a stack copy of geo, which waited
    // for every outstanding load
    const bool more = c.st + 1 < geo.hi;
    const bool cg_wrap = c.cg + 1 == geo.CG;
    const bool s_wrap = c.s + 1 == geo.S;
    const int inc = cg_wrap ? (s_wrap ? geo.d_r : geo.d_s) : geo.d_cg;
    const int cg_next = cg_wrap ? 0 : c.cg + 1;
    const int s_next = cg_wrap ? (s_wrap ? 0 : c.s + 1) : c.s;
    c.uoff = more ? c.uoff + inc : c.uoff;
    c.cg = more ? cg_next : c.cg;
    c.s = more ? s_next : c.s;
    c.st = more ? c.st + 1 : c.st;
}

// Output modes: the float32 epilogue, the raw int32 sums, the float32
// epilogue requantized to int8 into the next layer's halo'd input, or both
// the float32 output and its requantized copy; kOutDyn (group launches,
// whose members differ) writes whichever of y and yq is not null.
constexpr int kOutF32 = 0, kOutAcc = 1, kOutI8 = 2, kOutBoth = 3, kOutDyn = 4;

// One output tile u (channel tile kt, pixel tile pxt, pixel tiles fastest)
// of the convolution a, by all WAVES waves of the workgroup (wave: this
// wave's index, uniform; lane: its lane).
template <int FK, int FP, int WAVES, int MODE>
__device__ __forceinline__ void i8_tile(const I8Args& a, const int u, const int wave, const int lane) {
    const int li = lane & 15, g = lane >> 4;
    const int ohw = a.OH * a.OW;
    const int plane = a.Hp * a.Wp * 16;  // bytes per channel-block plane
    const int kt = fdiv(u, a.div_npx);
    const int pxt = u - kt * a.npx;

    bool pv[FP];
    int xbase[FP], obase[FP], ybase[FP], qbase[FP];
#pragma unroll
    for (int p = 0; p < FP; ++p) {
        const int m = (pxt * FP + p) * 16 + li;
        pv[p] = m < a.M;  // lanes past the last pixel compute pixel 0 and never store
        const int mm = pv[p] ? m : 0;
        const int n = fdiv(mm, a.div_ohw);
        const int pix = mm - n * ohw;
        const int oh = fdiv(pix, a.div_ow);
        const int ow = pix - oh * a.OW;
        // the (r, s) = (0, 0) byte of the pixel's window in channel block g
        xbase[p] = ((n * a.CB + g) * a.Hp + oh * a.sh + a.hoff) * a.Wp * 16 + (ow * a.sw + a.woff) * 16;
        // its output element in channel block 0 of [N][KB][OH][OW][16]
        // (residual, accumulators) and of the view: [N][y_tot][OH][OW][16]
        // float32, or in int8 mode [N][y_tot][OH + 2 qph][OW + 2 qpw][16]
        obase[p] = (n * a.KB * ohw + pix) * 16 + 4 * g;
        ybase[p] = (n * a.y_tot * ohw + pix) * 16 + 4 * g;
        const int owq = a.OW + 2 * a.qpw;
        qbase[p] = ((n * a.q_tot * (a.OH + 2 * a.qph) + oh + a.qph) * owq + ow + a.qpw) * 16 + 4 * g;
    }
    unsigned woff[FK];
#pragma unroll
    for (int f = 0; f < FK; ++f)
        woff[f] = (unsigned)((kt * FK + f) * a.T * 1024 + (g * 16 + li) * 16);

    // this wave's contiguous run of steps st = (r * S + s) * CG + cg
    const int w_lo = __builtin_amdgcn_readfirstlane((int)(((long)a.T * wave) / WAVES));
    const int w_hi = __builtin_amdgcn_readfirstlane((int)(((long)a.T * (wave + 1)) / WAVES));

    v4i acc[FK][FP];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int p = 0; p < FP; ++p) acc[f][p] = v4i{0, 0, 0, 0};

    // The step the next load reads, kept in scalar registers and advanced by
    // one per load (no divisions in the loop).  It stops at the run's last
    // step: loads past the run read that step again (never used), so every
    // load is unconditional and the waits count outstanding loads exactly.
    StepCursor cur;
    cur.st = w_lo;
    {
        const int rs = w_lo / a.CG;
        cur.cg = w_lo - rs * a.CG;
        const int r = rs / a.S;
        cur.s = rs - r * a.S;
        cur.uoff = cur.cg * 4 * plane + (r * a.Wp + cur.s) * 16;
    }
    const StepGeometry geo{a.CG, a.S, w_hi, 4 * plane, 16 - (a.CG - 1) * 4 * plane,
                           (a.Wp - a.S + 1) * 16 - (a.CG - 1) * 4 * plane};
    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a.x), (short)0, a.x_bytes, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t wr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int8_t*>(a.w), (short)0, a.w_bytes, kRsrcWord3);
    const int glim = a.CB - g;  // lane group g holds a real block while 4 cg < CB - g
#define NEO_I8_LOAD(A, B) load_step<FK, FP>(xr, wr, xbase, woff, glim, geo, cur, A, B)

    // two operand sets: the loads of step q + 1 are in flight during the
    // MFMAs of step q
    if (w_lo < w_hi) {
        v4i A0[FK], B0[FP], A1[FK], B1[FP];
        NEO_I8_LOAD(A0, B0);
        int st = w_lo;
        for (; st + 2 <= w_hi; st += 2) {
            NEO_I8_LOAD(A1, B1);
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A0[f], B0[p], acc[f][p], 0, 0, 0);
            NEO_I8_LOAD(A0, B0);
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A1[f], B1[p], acc[f][p], 0, 0, 0);
        }
        if (st < w_hi) {
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_i32_16x16x64_i8(A0[f], B0[p], acc[f][p], 0, 0, 0);
        }
    }

#undef NEO_I8_LOAD

    if constexpr (WAVES > 1) {
        __shared__ v4i red[WAVES - 1][FK * FP][64];
        if (wave > 0) {
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p) red[wave - 1][f * FP + p][lane] = acc[f][p];
        }
        __syncthreads();
        if (wave == 0) {
            // one partner wave at a time: all LDS reads hoisted at once would
            // need a register tile per partner
#pragma unroll 1
            for (int w = 0; w < WAVES - 1; ++w)
#pragma unroll
                for (int f = 0; f < FK; ++f)
#pragma unroll
                    for (int p = 0; p < FP; ++p) acc[f][p] += red[w][f * FP + p][lane];
        }
        // the partners may overwrite red for the next tile once wave 0 has it
        __syncthreads();
        if (wave != 0) return;
    }

    if constexpr (MODE == kOutAcc) {
#pragma unroll
        for (int f = 0; f < FK; ++f) {
            const int kofs = (kt * FK + f) * ohw * 16;
#pragma unroll
            for (int p = 0; p < FP; ++p)
                if (pv[p]) *reinterpret_cast<v4i*>(a.acc + obase[p] + kofs) = acc[f][p];
        }
        return;
    }
    const bool out_f32 = MODE == kOutF32 || MODE == kOutBoth || (MODE == kOutDyn && a.y);
    const bool out_i8 = MODE == kOutI8 || MODE == kOutBoth || (MODE == kOutDyn && a.yq);
    const bool relu = a.act == NEO_ACT_RELU;
    const int yofs = a.y_off * ohw * 16;
    const int qplane = (a.OH + 2 * a.qph) * (a.OW + 2 * a.qpw);  // one block of the int8 copy
#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kt * FK + f;
        const v4f ws = *reinterpret_cast<const v4f*>(a.wscale + kb * 16 + 4 * g);
        const v4f bb = a.bias ? *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * g) : v4f{0.f, 0.f, 0.f, 0.f};
        v4f mult;
#pragma unroll
        for (int v = 0; v < 4; ++v) mult[v] = a.xscale * ws[v];
        const int kofs = kb * ohw * 16;
#pragma unroll
        for (int p = 0; p < FP; ++p) {
            if (!pv[p]) continue;
            // ((acc * m) + b) + r, each operation rounded to float32 in this
            // order (no fused multiply-add): the value the interface defines
            v4f o;
            {
#pragma clang fp contract(off)
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = (float)acc[f][p][v] * mult[v];
                if (a.bias) o = o + bb;
                if (a.res) o = o + *reinterpret_cast<const v4f*>(a.res + obase[p] + kofs);
            }
            if (relu) {
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
            }
            if (out_f32) *reinterpret_cast<v4f*>(a.y + ybase[p] + yofs + kofs) = o;
            if (out_i8) {
                // clamp(round_half_even(y * (1 / s_y)), -127, 127), four
                // channels packed into one 4-byte store
                unsigned packed = 0;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    float q;
                    {
#pragma clang fp contract(off)
                        q = a.ydiv > 0.f ? rintf(o[v] / a.ydiv) : rintf(o[v] * a.yrcp);
                    }
                    q = q > (float)kQMax ? (float)kQMax : (q < -(float)kQMax ? -(float)kQMax : q);
                    packed |= ((unsigned)(int)q & 0xffu) << (8 * v);
                }
                *reinterpret_cast<unsigned*>(a.yq + qbase[p] + (a.q_off + kb) * qplane * 16) = packed;
            }
        }
    }
}

// Output tiles u = first, first + grid, ...: a workgroup runs several in
// turn, so the stores of one drain while the next one loads and multiplies.
// Pixel tiles fastest in each XCD's contiguous run (as the fp32 kernel below
// its large-launch threshold).
template <int FK, int FP, int WAVES, int MODE>
__global__ __launch_bounds__(WAVES * 64) void conv_i8(I8Args a) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int u = __builtin_amdgcn_readfirstlane(xcd_order()); u < a.ntiles; u += gridDim.x)
        i8_tile<FK, FP, WAVES, MODE>(a, u, wave, lane);
}

// Several independent integer convolutions in one launch (the float32 group
// launch's scheme, for batch 1, where each alone is too small to fill the
// chip): member m owns workgroups [start[m], start[m + 1]), a whole number of
// rounds over the XCDs, one tile per workgroup (cnt[m] real, the rest exit),
// its tiles in a launch of its own's per-XCD order.  Members share the tile
// and wave count and may differ in their outputs.  A pooling step may ride
// along in the workgroups past the convs' (the pooling kernel's arithmetic).
constexpr int kMaxI8Group = 4;
struct I8GroupArgs {
    I8Args a[kMaxI8Group];
    int start[kMaxI8Group + 1];
    int cnt[kMaxI8Group];
    int n;
    conv_detail::PoolPart pool;
};

template <int FK, int FP, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void conv_i8_group(I8GroupArgs ga) {
    const int nconv = ga.start[ga.n];
    if ((int)blockIdx.x >= nconv) {
        using conv_detail::pool_part_run;
        const int wg = blockIdx.x - nconv;
        if (ga.pool.max)
            ga.pool.k33 ? pool_part_run<true, 3, true>(ga.pool, wg) : pool_part_run<true, 0, true>(ga.pool, wg);
        else
            ga.pool.k33 ? pool_part_run<false, 3, true>(ga.pool, wg) : pool_part_run<false, 0, true>(ga.pool, wg);
        return;
    }
    int m = 0;
    while (m + 1 < ga.n && (int)blockIdx.x >= ga.start[m + 1]) ++m;
    m = __builtin_amdgcn_readfirstlane(m);
    const int b = blockIdx.x - ga.start[m];
    if (b >= ga.cnt[m]) return;
    i8_tile<FK, FP, WAVES, kOutDyn>(ga.a[m], xcd_order(b, ga.cnt[m]),
                                    __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), threadIdx.x & 63);
}

// fp32 NCHW16c [N][CB][H][W][16] -> int8 NCHW16c with a zero halo
// [N][CB][H + 2 ph][W + 2 pw][16]: clamp(round_half_even(x / scale), -127,
// 127), one pixel block (16 values) per thread.  Padding lanes (+0.0) give 0.
__global__ __launch_bounds__(256) void quantize_kernel(const float* x, int H, int W, int ph, int pw, long blocks,
                                                       float scale, int8_t* q) {
    const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= blocks) return;
    const int Wp = W + 2 * pw, Hp = H + 2 * ph;
    const long rowp = t / Wp;
    const int iw = (int)(t - rowp * Wp) - pw;
    const long plane = rowp / Hp;  // n * CB + cb
    const int ih = (int)(rowp - plane * Hp) - ph;
    union {
        int8_t b[16];
        v4i v;
    } out;
    out.v = v4i{0, 0, 0, 0};
    if ((unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W) {
        const v4f* src = reinterpret_cast<const v4f*>(x + ((plane * H + ih) * W + iw) * 16);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const v4f v = src[i];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                float r = rintf(v[j] / scale);
                r = r > (float)kQMax ? (float)kQMax : (r < -(float)kQMax ? -(float)kQMax : r);
                out.b[4 * i + j] = (int8_t)(int)r;
            }
        }
    }
    *reinterpret_cast<v4i*>(q + t * 16) = out.v;
}

// max |x| over n floats (n a multiple of 4, 16-byte aligned) into *out as
// the float's bits (non-negative floats order like their bit patterns): a
// grid-stride float4 pass (the last n % 4 floats by the first threads), a
// wave maximum, one vector atomic per wave.  *out must hold 0 before
// (absmax_clear).
__global__ __launch_bounds__(256) void absmax_kernel(const float* x, long n, unsigned* out) {
    float m = 0.f;
    const long n4 = n / 4;
    const long t0 = (long)blockIdx.x * blockDim.x + threadIdx.x;
    for (long i = t0; i < n4; i += (long)gridDim.x * blockDim.x) {
        const v4f v = reinterpret_cast<const v4f*>(x)[i];
        m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    }
    if (t0 < n - 4 * n4) m = fmaxf(m, fabsf(x[4 * n4 + t0]));
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
    if ((threadIdx.x & 63) == 0) atomicMax(out, __float_as_uint(m));
}

__global__ void absmax_clear(unsigned* out) {
    if (threadIdx.x == 0) *out = 0u;
}

// KCRS fp32 -> per-output-channel scales and the packed int8 filter, one
// workgroup per (padded) output channel: max |w[k]| by a tree in LDS, then
// every element quantized and written to its packed position.
__global__ __launch_bounds__(256) void pack_filter_i8_kernel(const float* w, int K, int C, int R, int S,
                                                             int8_t* wq, float* wscale) {
    const int k = blockIdx.x;
    const int CG = (C + 63) / 64;
    const long per = (long)C * R * S;
    __shared__ float red[256];
    float m = 0.f;
    if (k < K)
        for (long i = threadIdx.x; i < per; i += 256) m = fmaxf(m, fabsf(w[k * per + i]));
    red[threadIdx.x] = m;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + h]);
        __syncthreads();
    }
    const float mx = red[0];
    const float s = mx > 0.f ? mx / (float)kQMax : 1.f;
    if (threadIdx.x == 0) wscale[k] = s;
    // every (c, r, s) of this output channel's packed blocks, padding channels 0
    const long total = (long)CG * 64 * R * S;
    const int kb = k >> 4, kk = k & 15;
    for (long i = threadIdx.x; i < total; i += 256) {
        const int c = (int)(i / (R * S));
        const int rs = (int)(i - (long)c * R * S);
        const int r = rs / S, sx = rs - r * S;
        int8_t q = 0;
        if (k < K && c < C) {
            float v = rintf(w[(k * (long)C + c) * R * S + rs] / s);
            v = v > (float)kQMax ? (float)kQMax : (v < -(float)kQMax ? -(float)kQMax : v);
            q = (int8_t)(int)v;
        }
        const int cg = c >> 6, gg = (c >> 4) & 3, b = c & 15;
        wq[((((long)kb * R + r) * S + sx) * CG + cg) * 1024 + (gg * 16 + kk) * 16 + b] = q;
    }
}

// Integer dense layer (the fully connected layers of integer inference):
// acc[n][k] = sum_i xq[n][i] * wq[k][i], exact in int32 (|acc| <= 127^2 * IN),
// then the conv's float32 epilogue.  Rows of xq and wq are padded with zeros
// to INp = 16 * in16 bytes.  One wave per R output rows k0 .. k0 + R - 1:
// its lanes take the rows' 16-byte chunks in turn (one load per row and
// image, four 4-byte dot products per row and image), keep one sum per row
// and image, and add them across the wave; lane n then finishes image
// n0 + n of each row.  Images n0 .. n0 + NB - 1 per launch.  (R > 1 would
// reuse each input chunk for R rows; measured slower at 32 images than the
// 1x1 integer conv a plan runs there, so the launcher uses R = 1.)
struct DenseI8Args {
    const int8_t* x;      // [N][INp]
    const int8_t* w;      // [OUT][INp]
    const float* wscale;  // [OUT]
    float xscale;
    const float* bias;    // [OUT] or null
    float* y;             // [N][OUT] or null
    int8_t* yq;           // [N][OUTq] or null: y requantized by yrcp
    float yrcp;
    int N, in16, OUT, OUTq, act, n0;
};

template <int NB, int R>
__global__ __launch_bounds__(256) void dense_i8(DenseI8Args a) {
    const int lane = threadIdx.x & 63;
    const int k0 = (blockIdx.x * 4 + (threadIdx.x >> 6)) * R;
    if (k0 >= a.OUT) return;
    const long inp = 16L * a.in16;
    int acc[R][NB];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int n = 0; n < NB; ++n) acc[r][n] = 0;
    const int nb = min(NB, a.N - a.n0);
    // rows past OUT (the last wave of a ragged OUT) read row k0 again and are never stored
    const v4i* wr[R];
#pragma unroll
    for (int r = 0; r < R; ++r) wr[r] = reinterpret_cast<const v4i*>(a.w + (k0 + r < a.OUT ? k0 + r : k0) * inp);
    for (int c = lane; c < a.in16; c += 64) {
        v4i wv[R];
#pragma unroll
        for (int r = 0; r < R; ++r) wv[r] = wr[r][c];
#pragma unroll
        for (int n = 0; n < NB; ++n) {
            if (n < nb) {
                const v4i xv = reinterpret_cast<const v4i*>(a.x + (a.n0 + n) * inp)[c];
#pragma unroll
                for (int r = 0; r < R; ++r)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[r][n] = __builtin_amdgcn_sdot4(wv[r][j], xv[j], acc[r][n], false);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int n = 0; n < NB; ++n)
#pragma unroll
            for (int d = 32; d > 0; d >>= 1) acc[r][n] += __shfl_xor(acc[r][n], d, 64);
    if (lane >= nb) return;
    const int img = a.n0 + lane;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int k = k0 + r;
        if (k >= a.OUT) break;
        // lane n keeps image n's sum (a select chain, not a dynamic register index)
        int mine = acc[r][0];
#pragma unroll
        for (int n = 1; n < NB; ++n) mine = lane == n ? acc[r][n] : mine;
        float o;
        {
#pragma clang fp contract(off)
            const float m = a.xscale * a.wscale[k];
            o = (float)mine * m;
            if (a.bias) o = o + a.bias[k];
        }
        if (a.act == NEO_ACT_RELU) o = o > 0.f ? o : 0.f;
        if (a.y) a.y[(long)img * a.OUT + k] = o;
        if (a.yq) {
            float q;
            {
#pragma clang fp contract(off)
                q = rintf(o * a.yrcp);
            }
            q = q > (float)kQMax ? (float)kQMax : (q < -(float)kQMax ? -(float)kQMax : q);
            a.yq[(long)img * a.OUTq + k] = (int8_t)(int)q;
        }
    }
}

// float32 [N][IN] -> int8 [N][INp] (the padding bytes i >= IN written 0):
// clamp(round_half_even(x / scale), -127, 127), the division in float32.
__global__ __launch_bounds__(256) void quantize_rows_kernel(const float* x, long total, int IN, long inp,
                                                            float scale, int8_t* q) {
    const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;  // over N * INp
    if (t >= total) return;
    const long n = t / inp;
    const int i = (int)(t - n * inp);
    int8_t b = 0;
    if (i < IN) {
        float r = rintf(x[n * IN + i] / scale);
        r = r > (float)kQMax ? (float)kQMax : (r < -(float)kQMax ? -(float)kQMax : r);
        b = (int8_t)(int)r;
    }
    q[t] = b;
}

// A conv over few input channels (a network's stem) as a 1x1 conv: the
// float32 NCHW16c input [N][ceil(C/16)][H][W][16] quantized into its im2col
// rows, int8 NCHW16c [N][ceil(R*S*C/16)][OH][OW][16] with channel
// (r * S + s) * C + c holding input channel c at tap (r, s) of output pixel
// (oh, ow) (0 outside the image and past R*S*C), clamp(round_half_even(x /
// scale), -127, 127) with the division in float32.  The 1x1 conv over it
// sums the same products as the conv.  NCHW: the input is plain NCHW
// [N][C][H][W] instead (a network's input, read without its blocked copy).
//
// One workgroup per 64 output pixels of one row: the R input rows they
// read, span = 63 sw + S pixels wide, quantized once into LDS as int8 rows
// [C][R][span] plus one zero row (each input value is read by up to
// R S / (sh sw) taps; one float32 division per value), and a table of each
// im2col channel's offset in that tile (the zero row past R*S*C); then every
// thread assembles 16-byte output blocks with 16 LDS byte reads at its
// pixel's offset plus the table's (wave-uniform) entries.  64 consecutive
// pixels of a block row are one contiguous 1 KiB store.  No integer
// division per element: each thread steps its (row, column) by the
// workgroup size.
constexpr int kIm2colPix = 64;
template <bool NCHW>
__global__ __launch_bounds__(256) void im2col_q_kernel(const float* x, int C, int H, int W, int R, int S, int sh,
                                                       int sw, int ph, int pw, int OH, int OW, int CBc,
                                                       float scale, int8_t* q) {
    extern __shared__ int lds_words[];
    const int span = (kIm2colPix - 1) * sw + S;
    const int rows = C * R;                     // + the zero row
    int* table = lds_words;                     // [CBc * 16]
    int8_t* tile = reinterpret_cast<int8_t*>(lds_words + CBc * 16);  // [rows + 1][span]
    const int n = blockIdx.z, oh = blockIdx.y, ow0 = blockIdx.x * kIm2colPix;
    const int ih0 = oh * sh - ph, iw0 = ow0 * sw - pw;
    const int CBx = (C + 15) / 16;
    const float* xn = x + (NCHW ? (long)n * C * H * W : (long)n * CBx * H * W * 16);
    const int RSC = R * S * C;
    for (int ch = threadIdx.x; ch < CBc * 16; ch += 256) {  // (256 threads)
        int off = rows * span;                              // the zero row
        if (ch < RSC) {
            const int rs = ch / C, c = ch - rs * C, r = rs / S;
            off = (c * R + r) * span + (rs - r * S);
        }
        table[ch] = off;
    }
    // element e = row * span + j of the tile, row = c * R + r; thread t takes
    // e = t, t + 256, ...: (row, j) and (c, r) stepped, not divided
    const int total = (rows + 1) * span;
    const int drow = 256 / span, dj = 256 - drow * span;
    int j = threadIdx.x % span, r = threadIdx.x / span, c = 0;
    while (r >= R) {
        r -= R;
        ++c;
    }
    constexpr int kBatch = 8;  // loads in flight per thread before the first LDS store
    for (int e0 = threadIdx.x; e0 < total; e0 += kBatch * 256) {
        float v[kBatch];
        int slot[kBatch];
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            const int ih = ih0 + r, iw = iw0 + j;
            v[k] = (c < C && (unsigned)ih < (unsigned)H && (unsigned)iw < (unsigned)W)
                       ? (NCHW ? xn[((long)c * H + ih) * W + iw]
                               : xn[((long)((c >> 4) * H + ih) * W + iw) * 16 + (c & 15)])
                       : 0.f;
            slot[k] = (c * R + r) * span + j;  // = e0 + 256 k while inside the tile
            j += dj;
            r += drow;
            if (j >= span) {
                j -= span;
                ++r;
            }
            while (r >= R) {
                r -= R;
                ++c;
            }
        }
#pragma unroll
        for (int k = 0; k < kBatch; ++k) {
            float q8 = rintf(v[k] / scale);
            q8 = q8 > (float)kQMax ? (float)kQMax : (q8 < -(float)kQMax ? -(float)kQMax : q8);
            if (e0 + k * 256 < total) tile[slot[k]] = (int8_t)(int)q8;
        }
    }
    __syncthreads();
    const int owl = threadIdx.x % kIm2colPix, ow = ow0 + owl;
    if (ow >= OW) return;
    const int8_t* px = tile + owl * sw;
    for (int cb = threadIdx.x / kIm2colPix; cb < CBc; cb += 256 / kIm2colPix) {
        const int* t16 = table + cb * 16;
        union {
            int8_t b[16];
            v4i v;
        } out;
#pragma unroll
        for (int i = 0; i < 16; ++i) out.b[i] = px[t16[i]];
        *reinterpret_cast<v4i*>(q + ((((long)n * CBc + cb) * OH + oh) * OW + ow) * 16) = out.v;
    }
}

// The exit of the blocked layout for an integer dense layer: NCHW16c float32
// -> the flattened NCHW order, as float32 (y, may be null) and/or int8 rows
// (yq [N][inp]) quantized by division.  One thread per output element.
__global__ __launch_bounds__(256) void blk_to_rows_q(const float* x, int C, int H, int W, long total, long per,
                                                     long inp, float* y, int8_t* yq, float scale) {
    const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= total) return;
    const long n = t / per;
    const int i = (int)(t - n * per);  // (c * H + h) * W + w
    const int c = i / (H * W), hw = i - c * (H * W);
    const float v = x[((n * ((C + 15) / 16) + c / 16) * (long)(H * W) + hw) * 16 + (c & 15)];
    if (y) y[t] = v;
    if (yq) {
        float r = rintf(v / scale);
        r = r > (float)kQMax ? (float)kQMax : (r < -(float)kQMax ? -(float)kQMax : r);
        yq[n * inp + i] = (int8_t)(int)r;
    }
}

// A dense layer's weights [OUT][IN] float32 -> per-row scales max|w[k]| / 127
// (1 for a zero row) and int8 rows [OUT][INp] (padding 0), one workgroup per row.
__global__ __launch_bounds__(256) void pack_dense_i8_kernel(const float* w, int IN, long inp, int8_t* wq,
                                                            float* wscale) {
    const int k = blockIdx.x;
    __shared__ float red[256];
    float m = 0.f;
    for (long i = threadIdx.x; i < IN; i += 256) m = fmaxf(m, fabsf(w[(long)k * IN + i]));
    red[threadIdx.x] = m;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if ((int)threadIdx.x < h) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + h]);
        __syncthreads();
    }
    const float mx = red[0];
    const float s = mx > 0.f ? mx / (float)kQMax : 1.f;
    if (threadIdx.x == 0) wscale[k] = s;
    for (long i = threadIdx.x; i < inp; i += 256) {
        int8_t q = 0;
        if (i < IN) {
            float v = rintf(w[(long)k * IN + i] / s);
            v = v > (float)kQMax ? (float)kQMax : (v < -(float)kQMax ? -(float)kQMax : v);
            q = (int8_t)(int)v;
        }
        wq[(long)k * inp + i] = q;
    }
}

template <int FK, int FP, int WAVES, int MODE>
hipError_t launch_t(const I8Args& a, hipStream_t st) {
    // one workgroup per tile up to two rounds of the chip's SIMDs, then each
    // workgroup takes several tiles in turn
    const long cap = 2L * 1024 / WAVES;
    const long wgs = a.ntiles <= cap ? a.ntiles : std::max(cap, (long)(a.ntiles + 3) / 4);
    hipLaunchKernelGGL((conv_i8<FK, FP, WAVES, MODE>), dim3((unsigned)wgs), dim3(WAVES * 64), 0, st, a);
    return hipGetLastError();
}

template <int FK, int FP, int MODE>
hipError_t by_waves(int waves, const I8Args& a, hipStream_t st) {
    switch (waves) {
        case 1: return launch_t<FK, FP, 1, MODE>(a, st);
        case 2: return launch_t<FK, FP, 2, MODE>(a, st);
        case 4: return launch_t<FK, FP, 4, MODE>(a, st);
        default: return hipErrorInvalidValue;
    }
}

template <int MODE>
hipError_t by_tile(const ConvConfig& c, const I8Args& a, hipStream_t st) {
    if (c.fk == 1 && c.fp == 1) return by_waves<1, 1, MODE>(c.waves, a, st);
    if (c.fk == 1 && c.fp == 2) return by_waves<1, 2, MODE>(c.waves, a, st);
    if (c.fk == 2 && c.fp == 1) return by_waves<2, 1, MODE>(c.waves, a, st);
    if (c.fk == 2 && c.fp == 2) return by_waves<2, 2, MODE>(c.waves, a, st);
    if (c.fk == 4 && c.fp == 2) return by_waves<4, 2, MODE>(c.waves, a, st);
    if (c.fk == 2 && c.fp == 4) return by_waves<2, 4, MODE>(c.waves, a, st);
    if (c.fk == 4 && c.fp == 4) return by_waves<4, 4, MODE>(c.waves, a, st);
    if (c.fk == 8 && c.fp == 2) return by_waves<8, 2, MODE>(c.waves, a, st);
    if (c.fk == 8 && c.fp == 4) return by_waves<8, 4, MODE>(c.waves, a, st);
    return hipErrorInvalidValue;
}

template <int FK, int FP>
hipError_t group_by_waves(int waves, const I8GroupArgs& ga, int wgs, hipStream_t st) {
    switch (waves) {
        case 1: hipLaunchKernelGGL((conv_i8_group<FK, FP, 1>), dim3(wgs), dim3(64), 0, st, ga); break;
        case 2: hipLaunchKernelGGL((conv_i8_group<FK, FP, 2>), dim3(wgs), dim3(128), 0, st, ga); break;
        case 4: hipLaunchKernelGGL((conv_i8_group<FK, FP, 4>), dim3(wgs), dim3(256), 0, st, ga); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t group_by_tile(const ConvConfig& c, const I8GroupArgs& ga, int wgs, hipStream_t st) {
    if (c.fk == 1 && c.fp == 1) return group_by_waves<1, 1>(c.waves, ga, wgs, st);
    if (c.fk == 1 && c.fp == 2) return group_by_waves<1, 2>(c.waves, ga, wgs, st);
    if (c.fk == 2 && c.fp == 1) return group_by_waves<2, 1>(c.waves, ga, wgs, st);
    if (c.fk == 2 && c.fp == 2) return group_by_waves<2, 2>(c.waves, ga, wgs, st);
    if (c.fk == 4 && c.fp == 2) return group_by_waves<4, 2>(c.waves, ga, wgs, st);
    if (c.fk == 2 && c.fp == 4) return group_by_waves<2, 4>(c.waves, ga, wgs, st);
    if (c.fk == 4 && c.fp == 4) return group_by_waves<4, 4>(c.waves, ga, wgs, st);
    if (c.fk == 8 && c.fp == 2) return group_by_waves<8, 2>(c.waves, ga, wgs, st);
    if (c.fk == 8 && c.fp == 4) return group_by_waves<8, 4>(c.waves, ga, wgs, st);
    return hipErrorInvalidValue;
}

// The kernel arguments of one integer conv (its shape, launch
// configuration, operands and outputs).
I8Args make_i8_args(const ConvShape& s, const ConvConfig& c, const int8_t* x, const int8_t* w,
                    const float* wscale, float xscale, const float* bias, const float* res, float* y,
                    int* acc, int8_t* yq, float yscale, int qph, int qpw, int xph, int xpw,
                    int q_off = -1, int q_tot = -1, bool ydivide = false) {
    I8Args a;
    a.x = x;
    a.w = w;
    a.wscale = wscale;
    a.xscale = xscale;
    a.bias = bias;
    a.res = res;
    a.y = y;
    a.acc = acc;
    a.yq = yq;
    a.yrcp = yq ? 1.0f / yscale : 0.f;
    a.ydiv = yq && ydivide ? yscale : 0.f;
    a.qph = qph;
    a.qpw = qpw;
    // the int8 output takes the view of s when it is the only output; beside
    // the float32 output it is a whole tensor of its own; or the view given
    a.q_off = q_off >= 0 ? q_off : y ? 0 : s.y_off;
    a.q_tot = q_tot >= 0 ? q_tot : y ? cdiv(s.K, 16) : s.y_tot;
    a.N = s.N;
    a.CB = cdiv(s.C, 16);
    a.CG = cdiv(s.C, 64);
    // x's halo (xph, xpw) >= the padding: the window of output (oh, ow)
    // starts hoff = xph - ph rows and woff = xpw - pw columns into it
    a.Hp = s.H + 2 * xph;
    a.Wp = s.W + 2 * xpw;
    a.hoff = xph - s.ph;
    a.woff = xpw - s.pw;
    a.KB = cdiv(s.K, 16);
    a.S = s.S;
    a.sh = s.sh;
    a.sw = s.sw;
    a.OH = s.OH;
    a.OW = s.OW;
    a.M = s.N * s.OH * s.OW;
    a.y_off = s.y_off;
    a.y_tot = s.y_tot;
    a.act = s.act;
    a.T = s.R * s.S * a.CG;
    a.npx = cdiv(a.M, 16 * c.fp);
    a.nkt = a.KB / c.fk;
    a.ntiles = a.npx * a.nkt;
    a.x_bytes = (int)int8_act_bytes(s.N, s.C, s.H, s.W, xph, xpw);
    a.w_bytes = (int)int8_filter_bytes(s.K, s.C, s.R, s.S);
    a.div_ohw = make_fastdiv((unsigned)(s.OH * s.OW));
    a.div_ow = make_fastdiv((unsigned)s.OW);
    a.div_npx = make_fastdiv((unsigned)a.npx);
    return a;
}

}  // namespace

size_t int8_filter_bytes(int K, int C, int R, int S) {
    return (size_t)cdiv(K, 16) * cdiv(C, 64) * R * S * 1024;
}

bool int8_config_valid(const ConvShape& s, const ConvConfig& c) {
    const int KB = cdiv(s.K, 16);
    const bool tile = (c.fk == 1 && (c.fp == 1 || c.fp == 2)) || (c.fk == 2 && c.fp <= 4 && c.fp != 3) ||
                      ((c.fk == 4 || c.fk == 8) && (c.fp == 2 || c.fp == 4));
    return tile && KB % c.fk == 0 && c.split == 1 && (c.waves == 1 || c.waves == 2 || c.waves == 4) &&
           s.R * s.S * cdiv(s.C, 64) >= c.waves;
}

// The register tile and waves with the most tiles that still give every SIMD
// work: larger tiles load fewer bytes per MFMA, more waves split short grids.
ConvConfig choose_int8_config(const ConvShape& s) {
    const int KB = cdiv(s.K, 16), MP = cdiv(s.N * s.OH * s.OW, 16);
    static const ConvConfig order[] = {{4, 4, 1, 1}, {2, 4, 1, 1}, {4, 2, 1, 1}, {2, 2, 1, 1},
                                       {2, 1, 1, 1}, {1, 2, 1, 1}, {1, 1, 1, 1}};
    for (const ConvConfig& c0 : order) {
        if (KB % c0.fk) continue;
        const long tiles = (long)cdiv(MP, c0.fp) * (KB / c0.fk);
        for (int wv : {1, 2, 4}) {
            const ConvConfig c{c0.fk, c0.fp, 1, wv};
            if (int8_config_valid(s, c) && tiles * wv >= 1024) return c;
        }
    }
    for (int wv : {4, 2, 1}) {
        const ConvConfig c{1, 1, 1, wv};
        if (int8_config_valid(s, c)) return c;
    }
    return ConvConfig{1, 1, 1, 1};
}

hipError_t launch_absmax(const float* x, long n, unsigned* out, hipStream_t st) {
    hipLaunchKernelGGL(absmax_clear, dim3(1), dim3(64), 0, st, out);
    const long n4 = n / 4;
    const long blocks = std::min<long>(2048, std::max<long>(1, (n4 + 255) / 256));
    hipLaunchKernelGGL(absmax_kernel, dim3((unsigned)blocks), dim3(256), 0, st, x, n, out);
    return hipGetLastError();
}

size_t int8_act_bytes(int N, int C, int H, int W, int ph, int pw) {
    return (size_t)N * cdiv(C, 16) * (H + 2 * ph) * (W + 2 * pw) * 16;
}

hipError_t launch_quantize_int8(const float* x, int N, int C, int H, int W, int ph, int pw, float scale,
                                int8_t* q, hipStream_t st) {
    const long blocks = (long)(int8_act_bytes(N, C, H, W, ph, pw) / 16);
    hipLaunchKernelGGL(quantize_kernel, dim3((unsigned)((blocks + 255) / 256)), dim3(256), 0, st, x, H, W, ph, pw,
                       blocks, scale, q);
    return hipGetLastError();
}

hipError_t launch_pack_filter_int8(const float* w, int K, int C, int R, int S, int8_t* wq, float* wscale,
                                   hipStream_t st) {
    hipLaunchKernelGGL(pack_filter_i8_kernel, dim3((unsigned)(cdiv(K, 16) * 16)), dim3(256), 0, st, w, K, C,
                       R, S, wq, wscale);
    return hipGetLastError();
}

hipError_t launch_conv_int8(const ConvShape& s, const ConvConfig& c, const int8_t* x, const int8_t* w,
                            const float* wscale, float xscale, const float* bias, const float* res,
                            float* y, int* acc, int8_t* yq, float yscale, int qph, int qpw,
                            hipStream_t st, int xph, int xpw) {
    if (xph < 0) xph = s.ph;
    if (xpw < 0) xpw = s.pw;
    if (!int8_config_valid(s, c) || xph < s.ph || xpw < s.pw) return hipErrorInvalidValue;
    const I8Args a = make_i8_args(s, c, x, w, wscale, xscale, bias, res, y, acc, yq, yscale, qph, qpw, xph, xpw);
    if (acc) return by_tile<kOutAcc>(c, a, st);
    if (yq) return y ? by_tile<kOutBoth>(c, a, st) : by_tile<kOutI8>(c, a, st);
    return by_tile<kOutF32>(c, a, st);
}

hipError_t launch_conv_int8_m(const I8Member& m, const ConvConfig& c, hipStream_t st) {
    if (!int8_config_valid(m.s, c) || m.xph < m.s.ph || m.xpw < m.s.pw || (!m.y && !m.yq))
        return hipErrorInvalidValue;
    const I8Args a = make_i8_args(m.s, c, m.x, m.w, m.wscale, m.xscale, m.bias, m.res, m.y, nullptr, m.yq,
                                  m.yscale, m.qph, m.qpw, m.xph, m.xpw, m.q_off, m.q_tot, m.ydivide);
    if (m.yq) return m.y ? by_tile<kOutBoth>(c, a, st) : by_tile<kOutI8>(c, a, st);
    return by_tile<kOutF32>(c, a, st);
}

static_assert(kMaxI8Group == kMaxGroupConvs, "group size");

bool int8_group_config_valid(const ConvShape* s, int n, const ConvConfig& c) {
    if (n < 1 || n > kMaxGroupConvs) return false;
    for (int i = 0; i < n; ++i)
        if (!int8_config_valid(s[i], c)) return false;
    return true;
}

// The largest register tile (then the most waves) for which the members'
// tiles together still give every SIMD work, as for a single conv.
ConvConfig choose_int8_group_config(const ConvShape* s, int n) {
    static const ConvConfig order[] = {{4, 4, 1, 1}, {2, 4, 1, 1}, {4, 2, 1, 1}, {2, 2, 1, 1},
                                       {2, 1, 1, 1}, {1, 2, 1, 1}, {1, 1, 1, 1}};
    for (const ConvConfig& c0 : order) {
        long tiles = 0;
        for (int i = 0; i < n; ++i)
            tiles += (long)cdiv(cdiv(s[i].N * s[i].OH * s[i].OW, 16), c0.fp) * (cdiv(s[i].K, 16) / c0.fk);
        for (int wv : {1, 2, 4}) {
            const ConvConfig c{c0.fk, c0.fp, 1, wv};
            if (int8_group_config_valid(s, n, c) && tiles * wv >= 1024) return c;
        }
    }
    for (int wv : {4, 2, 1}) {
        const ConvConfig c{1, 1, 1, wv};
        if (int8_group_config_valid(s, n, c)) return c;
    }
    return ConvConfig{1, 1, 1, 1};
}

hipError_t launch_conv_int8_group(const I8Member* mem, int n, const ConvConfig& c, const GroupPool* pool,
                                  hipStream_t st) {
    ConvShape shp[kMaxGroupConvs];
    for (int i = 0; i < n && i < kMaxGroupConvs; ++i) shp[i] = mem[i].s;
    if (!int8_group_config_valid(shp, n, c)) return hipErrorInvalidValue;
    if (pool && pool->s.xb != 16) return hipErrorInvalidValue;
    I8GroupArgs ga;
    ga.n = n;
    ga.start[0] = 0;
    // dispatch order: the members with the most reduction steps first (they
    // finish last), ties in the given order
    int order[kMaxI8Group];
    for (int i = 0; i < n; ++i) order[i] = i;
    auto steps = [&](int i) { return shp[i].R * shp[i].S * cdiv(shp[i].C, 64); };
    std::stable_sort(order, order + n, [&](int p, int q) { return steps(p) > steps(q); });
    long total_wgs = 0;
    for (int j = 0; j < n; ++j) {
        const I8Member& m = mem[order[j]];
        if ((!m.y && !m.yq) || m.xph < m.s.ph || m.xpw < m.s.pw) return hipErrorInvalidValue;
        ga.a[j] = make_i8_args(m.s, c, m.x, m.w, m.wscale, m.xscale, m.bias, m.res, m.y, nullptr, m.yq,
                               m.yscale, m.qph, m.qpw, m.xph, m.xpw, m.q_off, m.q_tot, m.ydivide);
        ga.cnt[j] = ga.a[j].ntiles;
        total_wgs += (long)cdiv(ga.cnt[j], conv_detail::kXcds) * conv_detail::kXcds;
        if (total_wgs >= (1L << 30)) return hipErrorInvalidValue;
        ga.start[j + 1] = ga.start[j] + cdiv(ga.cnt[j], conv_detail::kXcds) * conv_detail::kXcds;
    }
    for (int i = n; i < kMaxI8Group; ++i) {
        ga.a[i] = ga.a[n - 1];
        ga.cnt[i] = 0;
        ga.start[i + 1] = ga.start[n];
    }
    conv_detail::PoolPart& pp = ga.pool;
    pp = conv_detail::PoolPart{};
    if (pool) {
        const PoolShape& ps = pool->s;
        pp.x = pool->x;
        pp.y = pool->y;
        pp.s = ps;
        pp.CB = cdiv(ps.C, ps.xb);
        pp.lq = 2;  // log2(16 / 4): four channel quads per 16-channel block
        const long total = ((long)ps.N * pp.CB * ps.OH * ps.OW) << pp.lq;
        if (total >= (1L << 31)) return hipErrorInvalidValue;
        pp.total = (int)total;
        pp.max = pool->max ? 1 : 0;
        pp.k33 = ps.R == 3 && ps.S == 3;
        pp.q = pool->q;
        if ((!pp.y && !pp.q.yq) || (pp.q.yq && !(pp.q.scale > 0.f))) return hipErrorInvalidValue;
        // one output quad per thread, at most 1024 workgroups (then grid-stride)
        const long per = 64L * c.waves;
        pp.wgs = (int)std::min<long>(1024, std::max<long>(1, (total + per - 1) / per));
    }
    return group_by_tile(c, ga, ga.start[n] + pp.wgs, st);
}

size_t dense_i8_row_bytes(int IN) { return (size_t)cdiv(IN, 16) * 16; }

ConvShape im2col_shape(const ConvShape& s) {
    ConvShape t = s;
    t.C = s.C * s.R * s.S;
    t.H = s.OH;
    t.W = s.OW;
    t.R = t.S = t.sh = t.sw = 1;
    t.ph = t.pw = 0;
    return t;
}

size_t im2col_lds_bytes(const ConvShape& s) {
    return (size_t)cdiv(s.C * s.R * s.S, 16) * 64 + (size_t)(s.C * s.R + 1) * ((kIm2colPix - 1) * s.sw + s.S);
}

hipError_t launch_im2col_int8(const float* x, bool nchw, const ConvShape& s, float scale, int8_t* q,
                              hipStream_t st) {
    const int CBc = cdiv(s.C * s.R * s.S, 16);
    const size_t lds = im2col_lds_bytes(s);
    if (s.N <= 0 || s.N > 65535 || s.OH <= 0 || s.OH > 65535 || s.OW <= 0 || lds > kIm2colMaxLds ||
        !(scale > 0.f))
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(nchw ? im2col_q_kernel<true> : im2col_q_kernel<false>, dim3(cdiv(s.OW, kIm2colPix), s.OH, s.N),
                       dim3(256), lds, st, x, s.C, s.H, s.W, s.R, s.S, s.sh, s.sw, s.ph, s.pw, s.OH, s.OW, CBc,
                       scale, q);
    return hipGetLastError();
}

hipError_t launch_blk_to_rows_int8(const float* x, int N, int C, int H, int W, float* y, int8_t* yq,
                                   float scale, hipStream_t st) {
    const long per = (long)C * H * W, total = (long)N * per;
    if (total <= 0 || !x || (!y && !yq) || (yq && !(scale > 0.f))) return hipErrorInvalidValue;
    hipLaunchKernelGGL(blk_to_rows_q, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, x, C, H, W, total,
                       per, (long)dense_i8_row_bytes((int)per), y, yq, scale);
    return hipGetLastError();
}

hipError_t launch_pack_dense_int8(const float* w, int OUT, int IN, int8_t* wq, float* wscale, hipStream_t st) {
    if (OUT <= 0 || IN <= 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(pack_dense_i8_kernel, dim3((unsigned)OUT), dim3(256), 0, st, w, IN,
                       (long)dense_i8_row_bytes(IN), wq, wscale);
    return hipGetLastError();
}

hipError_t launch_quantize_rows_int8(const float* x, int N, int IN, float scale, int8_t* q, hipStream_t st) {
    const long inp = (long)dense_i8_row_bytes(IN), total = (long)N * inp;
    if (N <= 0 || IN <= 0 || !(scale > 0.f)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(quantize_rows_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, x, total, IN,
                       inp, scale, q);
    return hipGetLastError();
}

hipError_t launch_dense_int8(const int8_t* xq, const int8_t* wq, const float* wscale, float xscale,
                             const float* bias, int N, int IN, int OUT, int act, float* y, int8_t* yq,
                             float yscale, hipStream_t st) {
    if (N <= 0 || IN <= 0 || OUT <= 0 || (!y && !yq) || (long)IN * 127 * 127 >= (1L << 31))
        return hipErrorInvalidValue;
    DenseI8Args a;
    a.x = xq;
    a.w = wq;
    a.wscale = wscale;
    a.xscale = xscale;
    a.bias = bias;
    a.y = y;
    a.yq = yq;
    a.yrcp = yq ? 1.0f / yscale : 0.f;
    a.N = N;
    a.in16 = cdiv(IN, 16);
    a.OUT = OUT;
    a.OUTq = (int)dense_i8_row_bytes(OUT);
    a.act = act;
    // one row per wave: the weight stream bounds the layer for a few images
    // (a plan runs a dense layer over many images as a 1x1 integer conv)
    const dim3 g1((unsigned)cdiv(OUT, 4)), block(256);
    for (int n0 = 0; n0 < N; n0 += 32) {
        a.n0 = n0;
        const int nb = std::min(32, N - n0);
        if (nb == 1) hipLaunchKernelGGL((dense_i8<1, 1>), g1, block, 0, st, a);
        else if (nb == 2) hipLaunchKernelGGL((dense_i8<2, 1>), g1, block, 0, st, a);
        else if (nb <= 4) hipLaunchKernelGGL((dense_i8<4, 1>), g1, block, 0, st, a);
        else if (nb <= 8) hipLaunchKernelGGL((dense_i8<8, 1>), g1, block, 0, st, a);
        else if (nb <= 16) hipLaunchKernelGGL((dense_i8<16, 1>), g1, block, 0, st, a);
        else hipLaunchKernelGGL((dense_i8<32, 1>), g1, block, 0, st, a);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace neo
