// Two pointwise convolutions in one launch (vertical fusion; not in the
// paper): y = act_a(W_a x + b_a + r) and z = act_b(W_b y + b_b), both 1x1
// stride 1 on NCHW16c, where y is also stored (later layers read it, e.g. as
// a residual).  At batch 1 every launch costs about 3.5 us whatever its
// work, and a bottleneck's expanding 1x1 and the next bottleneck's reducing
// 1x1 at the 64-channel width are each a fraction of that.
//
// One workgroup per 16 output pixels holds all of y for those pixels:
//   phase 1  wave w computes y's channel groups [w*KPW, (w+1)*KPW) over the
//            whole reduction (C_a <= 64: every operand is loaded up front),
//            applies the epilogue, stores y and writes it to LDS as
//            [group][pixel][16 channels];
//   phase 2  wave w computes z's channel group w % K1B over the part
//            w / K1B of the reduction, its operand y read from LDS (the
//            filter loads are issued before the barrier); the parts are
//            summed in part order through LDS and the epilogue applied.
// Operand layouts and the MFMA mapping are the convolution kernel's
// (16x16x4 f32; lane = (pixel i, k-group g); filters in kernel order).
// Further down, the same two phases led by a 3x3 convolution (conv3x3_chain).
#include "neo_internal.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

struct PairArgs {
    const float *x, *wa, *ba, *res;
    float* y;
    const float *wb, *bb;
    float* z;
    int HW, M, act_a, act_b;
};

constexpr int kXcds = 8;

template <int WAVES, int CAB, int KAB, int KBB>
__global__ __launch_bounds__(WAVES * 64) void conv1x1_pair(PairArgs a) {
    constexpr int KPW = KAB / WAVES, P2 = WAVES / KBB, C2W = KAB / P2;
    static_assert(KAB % WAVES == 0 && WAVES % KBB == 0, "work split");
    extern __shared__ v4f lds[];  // y: KAB * 16 * 4 float4, then the phase-2 partial sums
    // XCD-aware order (workgroups are dispatched round-robin over the XCDs):
    // every XCD takes a contiguous run of pixel tiles
    const int nwg = gridDim.x, xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
    const int tile = xcd * (nwg / kXcds) + min(xcd, nwg % kXcds) + slot;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15, g = lane >> 4;
    const int m = tile * 16 + li;
    const bool pv = m < a.M;  // lanes past the last pixel compute on pixel 0 and store nothing
    const int mm = pv ? m : 0;
    const int n = mm / a.HW, pix = mm - n * a.HW;

    // every operand of both phases is requested before any is used
    v4f xb[CAB];
#pragma unroll
    for (int cb = 0; cb < CAB; ++cb)
        xb[cb] = *reinterpret_cast<const v4f*>(a.x + ((n * CAB + cb) * a.HW + pix) * 16 + 4 * g);
    v4f wa[KPW][CAB];
#pragma unroll
    for (int f = 0; f < KPW; ++f)
#pragma unroll
        for (int cb = 0; cb < CAB; ++cb)
            wa[f][cb] = *reinterpret_cast<const v4f*>(a.wa + ((wave * KPW + f) * CAB + cb) * 256 + (g * 16 + li) * 4);
    const int kt = wave % KBB, part = wave / KBB;
    v4f wb[C2W];
#pragma unroll
    for (int j = 0; j < C2W; ++j)
        wb[j] = *reinterpret_cast<const v4f*>(a.wb + (kt * KAB + part * C2W + j) * 256 + (g * 16 + li) * 4);
    v4f ba[KPW], rs[KPW];
#pragma unroll
    for (int f = 0; f < KPW; ++f) {
        const int kb = wave * KPW + f;
        ba[f] = a.ba ? *reinterpret_cast<const v4f*>(a.ba + kb * 16 + 4 * g) : v4f{0.f, 0.f, 0.f, 0.f};
        rs[f] = a.res && pv ? *reinterpret_cast<const v4f*>(a.res + ((n * KAB + kb) * a.HW + pix) * 16 + 4 * g)
                            : v4f{0.f, 0.f, 0.f, 0.f};
    }

    // phase 1: y for this wave's channel groups
    v4f acc[KPW];
#pragma unroll
    for (int f = 0; f < KPW; ++f) acc[f] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cb = 0; cb < CAB; ++cb)
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int f = 0; f < KPW; ++f)
                acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[f][cb][t], xb[cb][t], acc[f], 0, 0, 0);
#pragma unroll
    for (int f = 0; f < KPW; ++f) {
        const int kb = wave * KPW + f;
        v4f o = acc[f] + ba[f];
        o += rs[f];
        if (a.act_a == NEO_ACT_RELU) {
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
        }
        if (pv) *reinterpret_cast<v4f*>(a.y + ((n * KAB + kb) * a.HW + pix) * 16 + 4 * g) = o;
        lds[(kb * 16 + li) * 4 + g] = pv ? o : v4f{0.f, 0.f, 0.f, 0.f};
    }
    __syncthreads();

    // phase 2: z's channel group kt over part `part` of y's channel groups
    v4f acc2 = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < C2W; ++j) {
        const v4f yb = lds[((part * C2W + j) * 16 + li) * 4 + g];
#pragma unroll
        for (int t = 0; t < 4; ++t) acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(wb[j][t], yb[t], acc2, 0, 0, 0);
    }
    if constexpr (P2 > 1) {
        v4f* red = lds + KAB * 64;
        if (part > 0) red[((part - 1) * KBB + kt) * 64 + lane] = acc2;
        __syncthreads();
        if (part != 0) return;
#pragma unroll
        for (int q = 1; q < P2; ++q) acc2 += red[((q - 1) * KBB + kt) * 64 + lane];
    }
    v4f o = acc2 + (a.bb ? *reinterpret_cast<const v4f*>(a.bb + kt * 16 + 4 * g) : v4f{0.f, 0.f, 0.f, 0.f});
    if (a.act_b == NEO_ACT_RELU) {
#pragma unroll
        for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
    }
    if (pv) *reinterpret_cast<v4f*>(a.z + ((n * KBB + kt) * a.HW + pix) * 16 + 4 * g) = o;
}

template <int WAVES, int CAB, int KAB, int KBB>
hipError_t launch_pair_t(const PairArgs& a, hipStream_t st) {
    constexpr int P2 = WAVES / KBB;
    const size_t lds = (size_t)KAB * 1024 + (size_t)(P2 - 1) * KBB * 1024;
    hipLaunchKernelGGL((conv1x1_pair<WAVES, CAB, KAB, KBB>), dim3(cdiv(a.M, 16)), dim3(WAVES * 64), lds, st, a);
    return hipGetLastError();
}

// The channel-group counts (ceil(C_a/16), ceil(K_a/16), ceil(K_b/16)) with a
// kernel: 64 -> 256 -> 64 (inside a bottleneck stage) and 64 -> 256 -> 128
// (into the next stage's first reducing conv).
bool pair_blocks(int cab, int kab, int kbb) { return cab == 4 && kab == 16 && (kbb == 4 || kbb == 8); }

bool pointwise(const ConvShape& s) {
    return s.R == 1 && s.S == 1 && s.sh == 1 && s.sw == 1 && s.ph == 0 && s.pw == 0 && s.xb == 16 &&
           s.yb == 16 && !s.gap && s.y_off == 0 && s.y_tot == cdiv(s.K, 16);
}

// A 3x3 convolution followed by the pointwise expansion that reads its output
// and, optionally, the next pointwise reduction (the three convolutions of a
// ResNet bottleneck at the 64-channel width from its 3x3 on: 64 -> 64 3x3,
// 64 -> 256 1x1 with the residual, 256 -> 64 or 128 1x1), in one launch.  The
// 3x3's output is read by the expansion only and never stored.
//
// One workgroup (8 waves) per 16 output pixels:
//   phase 0  the 3x3's reduction is 36 (channel group, tap) blocks of 16
//            elements; wave w takes blocks w, w + 8, ... for all four output
//            groups (one input float4 and four filter float4s per block, all
//            requested up front; a tap outside the image reads 0 through the
//            buffer bounds).  The eight partial tiles are summed in wave order
//            through LDS, bias and activation applied, and the result kept in
//            LDS as the expansion's input operand;
//   phase 1  the expansion, as phase 1 of the pair kernel above;
//   phase 2  the reduction (KBB > 0), as phase 2 of the pair kernel.
struct ChainArgs {
    const float *x, *w0, *b0;  // 3x3: input (NCHW16c, 4 groups), filter in kernel order, bias
    const float *wa, *ba, *res;
    float* y;
    const float *wb, *bb;
    float* z;
    int H, W, HW, M, x_bytes, act0, act_a, act_b;
};

constexpr unsigned kRsrcWord3 = 0x00020000;    // raw buffer, gfx9 family
constexpr unsigned kOutOfRange = 0x80000000u;  // buffer offset that reads as 0

template <int KBB>
__global__ __launch_bounds__(512) void conv3x3_chain(ChainArgs a) {
    constexpr int WAVES = 8, CB0 = 4, KG0 = 4, CAB = 4, KAB = 16, KPW = KAB / WAVES;
    constexpr int NBLK = CB0 * 9, BPW = (NBLK + WAVES - 1) / WAVES;
    constexpr int P2 = KBB > 0 ? WAVES / KBB : 1, C2W = KAB / P2;
    static_assert(KBB == 0 || WAVES % KBB == 0, "work split");
    // phase-0 partial tiles [wave][group][lane]; then y as [group][pixel][16]
    // followed by the phase-2 partial sums
    __shared__ v4f red[WAVES * KG0 * 64];
    __shared__ v4f mid[KG0 * 64];  // the 3x3's output, [group][lane]
    const int nwg = gridDim.x, xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
    const int tile = xcd * (nwg / kXcds) + min(xcd, nwg % kXcds) + slot;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15, g = lane >> 4;
    const int m = tile * 16 + li;
    const bool pv = m < a.M;  // lanes past the last pixel compute on pixel 0 and store nothing
    const int mm = pv ? m : 0;
    const int n = mm / a.HW, pix = mm - n * a.HW;
    const int oh = pix / a.W, ow = pix - oh * a.W;

    const __amdgpu_buffer_rsrc_t xr =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.x), (short)0, a.x_bytes, kRsrcWord3);
    v4f x0[BPW], w0[BPW][KG0];
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
        const int blk = wave + j * WAVES;
        const bool bv = blk < NBLK;
        const int b = bv ? blk : 0;
        const int cb = b / 9, tap = b - cb * 9, r = tap / 3, sc = tap - r * 3;
        const int ih = oh + r - 1, iw = ow + sc - 1;
        const bool ok = bv && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
        const unsigned off = ok ? (unsigned)(((((n * CB0 + cb) * a.H + ih) * a.W + iw) * 16 + 4 * g) * 4)
                                : kOutOfRange;
        x0[j] = __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(xr, off, 0, 0));
#pragma unroll
        for (int kg = 0; kg < KG0; ++kg)
            w0[j][kg] = *reinterpret_cast<const v4f*>(a.w0 + ((kg * CB0 + cb) * 9 + tap) * 256 + (g * 16 + li) * 4);
    }
    v4f wa[KPW][CAB];
#pragma unroll
    for (int f = 0; f < KPW; ++f)
#pragma unroll
        for (int cb = 0; cb < CAB; ++cb)
            wa[f][cb] = *reinterpret_cast<const v4f*>(a.wa + ((wave * KPW + f) * CAB + cb) * 256 + (g * 16 + li) * 4);
    v4f ba[KPW], rs[KPW];
#pragma unroll
    for (int f = 0; f < KPW; ++f) {
        const int kb = wave * KPW + f;
        ba[f] = a.ba ? *reinterpret_cast<const v4f*>(a.ba + kb * 16 + 4 * g) : v4f{0.f, 0.f, 0.f, 0.f};
        rs[f] = a.res && pv ? *reinterpret_cast<const v4f*>(a.res + ((n * KAB + kb) * a.HW + pix) * 16 + 4 * g)
                            : v4f{0.f, 0.f, 0.f, 0.f};
    }

    // phase 0: this wave's part of the 3x3 for all four output groups
    v4f acc0[KG0];
#pragma unroll
    for (int kg = 0; kg < KG0; ++kg) acc0[kg] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < BPW; ++j) {
        if (wave + j * WAVES < NBLK) {  // uniform
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int kg = 0; kg < KG0; ++kg)
                    acc0[kg] = __builtin_amdgcn_mfma_f32_16x16x4f32(w0[j][kg][t], x0[j][t], acc0[kg], 0, 0, 0);
        }
    }
#pragma unroll
    for (int kg = 0; kg < KG0; ++kg) red[(wave * KG0 + kg) * 64 + lane] = acc0[kg];
    __syncthreads();
    if (wave < KG0) {
        const int kg = wave;
        v4f o = red[kg * 64 + lane];
#pragma unroll
        for (int q = 1; q < WAVES; ++q) o += red[(q * KG0 + kg) * 64 + lane];
        o += a.b0 ? *reinterpret_cast<const v4f*>(a.b0 + kg * 16 + 4 * g) : v4f{0.f, 0.f, 0.f, 0.f};
        if (a.act0 == NEO_ACT_RELU) {
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
        }
        mid[kg * 64 + lane] = o;
    }
    __syncthreads();

    // phase 1: the expansion's channel groups of this wave
    v4f acc[KPW];
#pragma unroll
    for (int f = 0; f < KPW; ++f) acc[f] = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int cb = 0; cb < CAB; ++cb) {
        const v4f xb = mid[cb * 64 + lane];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int f = 0; f < KPW; ++f)
                acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[f][cb][t], xb[t], acc[f], 0, 0, 0);
    }
    v4f* ylds = red;  // the phase-0 partials are all read (barrier above)
#pragma unroll
    for (int f = 0; f < KPW; ++f) {
        const int kb = wave * KPW + f;
        v4f o = acc[f] + ba[f];
        o += rs[f];
        if (a.act_a == NEO_ACT_RELU) {
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
        }
        if (pv) *reinterpret_cast<v4f*>(a.y + ((n * KAB + kb) * a.HW + pix) * 16 + 4 * g) = o;
        if constexpr (KBB > 0) ylds[(kb * 16 + li) * 4 + g] = o;
    }
    if constexpr (KBB > 0) {
        const int kt = wave % KBB, part = wave / KBB;
        v4f wb[C2W];
#pragma unroll
        for (int j = 0; j < C2W; ++j)
            wb[j] = *reinterpret_cast<const v4f*>(a.wb + (kt * KAB + part * C2W + j) * 256 + (g * 16 + li) * 4);
        __syncthreads();
        // phase 2: the reduction's channel group kt over part `part` of y's groups
        v4f acc2 = v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < C2W; ++j) {
            const v4f yb = ylds[((part * C2W + j) * 16 + li) * 4 + g];
#pragma unroll
            for (int t = 0; t < 4; ++t) acc2 = __builtin_amdgcn_mfma_f32_16x16x4f32(wb[j][t], yb[t], acc2, 0, 0, 0);
        }
        if constexpr (P2 > 1) {
            v4f* red2 = red + KAB * 64;
            if (part > 0) red2[((part - 1) * KBB + kt) * 64 + lane] = acc2;
            __syncthreads();
            if (part != 0) return;
#pragma unroll
            for (int q = 1; q < P2; ++q) acc2 += red2[((q - 1) * KBB + kt) * 64 + lane];
        }
        v4f o = acc2 + (a.bb ? *reinterpret_cast<const v4f*>(a.bb + kt * 16 + 4 * g) : v4f{0.f, 0.f, 0.f, 0.f});
        if (a.act_b == NEO_ACT_RELU) {
#pragma unroll
            for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
        }
        if (pv) *reinterpret_cast<v4f*>(a.z + ((n * KBB + kt) * a.HW + pix) * 16 + 4 * g) = o;
    }
}

template <int KBB>
hipError_t launch_chain_t(const ChainArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((conv3x3_chain<KBB>), dim3(cdiv(a.M, 16)), dim3(512), 0, st, a);
    return hipGetLastError();
}

bool chain_lead(const ConvShape& s) {
    return s.R == 3 && s.S == 3 && s.sh == 1 && s.sw == 1 && s.ph == 1 && s.pw == 1 && s.xb == 16 &&
           s.yb == 16 && !s.gap && cdiv(s.C, 16) == 4 && cdiv(s.K, 16) == 4 && s.OH == s.H && s.OW == s.W;
}

}  // namespace

bool conv_pair_eligible(const ConvShape& a, const ConvShape& b) {
    return pointwise(a) && pointwise(b) && a.K == b.C && a.N == b.N && a.OH == b.H && a.OW == b.W &&
           pair_blocks(cdiv(a.C, 16), cdiv(a.K, 16), cdiv(b.K, 16));
}

hipError_t launch_conv_pair(const ConvShape& sa, const ConvShape& sb, const float* x, const float* wa,
                            const float* ba, const float* res, float* y, const float* wb,
                            const float* bb, float* z, hipStream_t st) {
    if (!conv_pair_eligible(sa, sb)) return hipErrorInvalidValue;
    if ((long)sa.N * sa.OH * sa.OW * cdiv(sa.K, 16) * 16 >= (1L << 29)) return hipErrorInvalidValue;
    const PairArgs a{x, wa, ba, res, y, wb, bb, z, sa.OH * sa.OW, sa.N * sa.OH * sa.OW, sa.act, sb.act};
    if (cdiv(sb.K, 16) == 8) return launch_pair_t<8, 4, 16, 8>(a, st);
    return launch_pair_t<8, 4, 16, 4>(a, st);
}

bool conv_chain_eligible(const ConvShape* s, int n) {
    if (n < 2 || n > 3 || !chain_lead(s[0]) || !pointwise(s[1]) || s[1].C != s[0].K || s[1].N != s[0].N ||
        s[1].H != s[0].OH || s[1].W != s[0].OW || cdiv(s[1].K, 16) != 16)
        return false;
    return n == 2 || conv_pair_eligible(s[1], s[2]);
}

hipError_t launch_conv_chain(const ConvShape* s, int n, const float* x, const float* w0, const float* b0,
                             const float* wa, const float* ba, const float* res, float* y,
                             const float* wb, const float* bb, float* z, hipStream_t st) {
    if (!conv_chain_eligible(s, n)) return hipErrorInvalidValue;
    if ((long)s[1].N * s[1].OH * s[1].OW * 256 >= (1L << 29)) return hipErrorInvalidValue;
    const long x_bytes = (long)s[0].N * 64 * s[0].H * s[0].W * 4;
    const int HW = s[0].OH * s[0].OW;
    const ChainArgs a{x, w0, b0, wa, ba, res, y, wb, bb, z, s[0].H, s[0].W, HW, s[0].N * HW,
                      (int)x_bytes, s[0].act, s[1].act, n == 3 ? s[2].act : 0};
    if (n == 2) return launch_chain_t<0>(a, st);
    if (cdiv(s[2].K, 16) == 8) return launch_chain_t<8>(a, st);
    return launch_chain_t<4>(a, st);
}

}  // namespace neo
