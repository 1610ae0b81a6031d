// Layout-tolerant pooling on NCHW[x]c (Section 3.2): max, average, global
// average, for any block x of 4..64 channels.  One thread per (output pixel,
// 4-channel quad) moves float4s: the x/4 quads of a pixel block are
// neighbouring lanes, so a wave reads and writes 1 KB contiguous per access.
// Max pooling ignores taps outside the input (as if padded with -inf); average
// pooling divides by the number of taps inside it.
// Padded channel lanes hold 0 in the input and stay 0 in the output.
#include "pool_kernel.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

// One thread per output quad (pool_elem), grid-stride.
template <bool MAX, int KR, int KS>
__global__ __launch_bounds__(256) void pool_blk(const float* __restrict__ x, float* __restrict__ y,
                                                PoolShape s, int CB, int lq) {
    const int total = (s.N * CB * s.OH * s.OW) << lq;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x)
        pool_detail::pool_elem<MAX, KR, KS>(x, y, s, CB, lq, t);
}

// The same, on NCHW16c, with the int8 copy of the output (pool_elem's Q).
template <bool MAX, int KR, int KS>
__global__ __launch_bounds__(256) void pool_blk_q(const float* __restrict__ x, float* __restrict__ y,
                                                  PoolShape s, int CB, PoolQ q) {
    const int total = (s.N * CB * s.OH * s.OW) << 2;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x)
        pool_detail::pool_elem<MAX, KR, KS, true>(x, y, s, CB, 2, t, q);
}

// One wave per (n, 16-channel group j) whatever the block x: lane = 4 *
// pixel_slot + quad; each lane sums the pixels p = slot, slot + 16, ... of its
// quad's channels, then the 16 slots are summed with cross-lane shuffles in a
// fixed tree order -- the same order for every block, so the result does not
// depend on the layout.  The sums are in double and the mean is rounded once
// to float32: n float32 values whose exponents span e bits sum exactly in a
// double while n * 2^(e + 24) <= 2^53 (for a 7x7 or 8x8 map: nonzero values
// within a factor 2^23 of each other), and then the result is the exact mean
// rounded, whatever the order.  Channel c = 16 j + 4 q sits in block c / x at
// lane c % x (lx = log2 x); quads past the last block (x < 16) are idle.
// Q: the means also (or only: y null) written as int8 rows yq [N][inp]
// (block 16: channel c of image n at n * inp + c), clamp(round_half_even(
// mean / scale), -127, 127) with the division in float32.
template <bool Q>
__global__ __launch_bounds__(256) void gap_blk(const float* __restrict__ x, float* __restrict__ y,
                                               int N, int G16, int XB, int lx, int HW, int8_t* yq = nullptr,
                                               float scale = 1.f, int inp = 0) {
    const int wave_id = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (wave_id >= N * G16) return;
    const int n = wave_id / G16, j = wave_id - n * G16;
    const int lane = threadIdx.x & 63;
    const int q = lane & 3, slot = lane >> 2;
    const int X = 1 << lx;
    const int c = 16 * j + 4 * q;
    const bool ok = c < (XB << lx);
    const int blk = n * XB + (c >> lx), sub = c & (X - 1);
    const float* xb = x + (long)blk * HW * X + sub;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (ok) {
        int p = slot;
        for (; p + 48 < HW; p += 64) {  // four pixels of the slot in flight
            v4f v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const v4f*>(xb + (p + 16 * u) * X);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[i] += (double)v[u][i];
        }
        for (; p < HW; p += 16) {
            const v4f v = *reinterpret_cast<const v4f*>(xb + p * X);
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] += (double)v[i];
        }
    }
#pragma unroll
    for (int off = 4; off < 64; off <<= 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] += __shfl_xor(acc[i], off, 64);
    }
    if (slot == 0 && ok) {
        const double d = (double)HW;
        v4f o;
#pragma unroll
        for (int i = 0; i < 4; ++i) o[i] = (float)(acc[i] / d);
        if (!Q || y) *reinterpret_cast<v4f*>(y + blk * X + sub) = o;
        if constexpr (Q) {
            unsigned packed = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float r = rintf(o[i] / scale);
                r = r > 127.f ? 127.f : (r < -127.f ? -127.f : r);
                packed |= ((unsigned)(int)r & 0xffu) << (8 * i);
            }
            *reinterpret_cast<unsigned*>(yq + (long)n * inp + c) = packed;
        }
    }
}

inline dim3 grid_for(long total) {
    long b = (total + 255) / 256;
    if (b > 65536) b = 65536;
    if (b < 1) b = 1;
    return dim3((unsigned)b);
}

}  // namespace

template <bool MAX>
hipError_t launch_pool(const PoolShape& s, const float* x, float* y, hipStream_t st) {
    if (!pow2_block(s.xb) || !x || !y) return hipErrorInvalidValue;
    const int CB = cdiv(s.C, s.xb), lq = ilog2(s.xb / 4);
    const dim3 g = grid_for(((long)s.N * CB * s.OH * s.OW) << lq), b(256);
    if (s.R == 3 && s.S == 3)
        hipLaunchKernelGGL((pool_blk<MAX, 3, 3>), g, b, 0, st, x, y, s, CB, lq);
    else if (s.R == 2 && s.S == 2)
        hipLaunchKernelGGL((pool_blk<MAX, 2, 2>), g, b, 0, st, x, y, s, CB, lq);
    else
        hipLaunchKernelGGL((pool_blk<MAX, 0, 0>), g, b, 0, st, x, y, s, CB, lq);
    return hipGetLastError();
}

hipError_t launch_maxpool(const PoolShape& s, const float* x, float* y, hipStream_t st) {
    return launch_pool<true>(s, x, y, st);
}

hipError_t launch_avgpool(const PoolShape& s, const float* x, float* y, hipStream_t st) {
    return launch_pool<false>(s, x, y, st);
}

template <bool MAX>
hipError_t launch_pool_q_t(const PoolShape& s, const float* x, float* y, const PoolQ& q, hipStream_t st) {
    const int CB = cdiv(s.C, 16);
    const dim3 g = grid_for(((long)s.N * CB * s.OH * s.OW) << 2), b(256);
    if (s.R == 3 && s.S == 3)
        hipLaunchKernelGGL((pool_blk_q<MAX, 3, 3>), g, b, 0, st, x, y, s, CB, q);
    else if (s.R == 2 && s.S == 2)
        hipLaunchKernelGGL((pool_blk_q<MAX, 2, 2>), g, b, 0, st, x, y, s, CB, q);
    else
        hipLaunchKernelGGL((pool_blk_q<MAX, 0, 0>), g, b, 0, st, x, y, s, CB, q);
    return hipGetLastError();
}

hipError_t launch_pool_q(const PoolShape& s, bool max, const float* x, float* y, const PoolQ& q,
                         hipStream_t st) {
    if (s.xb != 16 || !x || (!y && !q.yq) || (q.yq && !(q.scale > 0.f))) return hipErrorInvalidValue;
    return max ? launch_pool_q_t<true>(s, x, y, q, st) : launch_pool_q_t<false>(s, x, y, q, st);
}

// One thread per output pixel block: the byte-wise max over the window's
// in-image taps (a window always holds one), one 16-byte store.
__global__ __launch_bounds__(256) void maxpool_i8_blk(const int8_t* __restrict__ x, PoolShape s, int CB, PoolQ q) {
    const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (long)s.N * CB * s.OH * s.OW) return;
    const int ow = (int)(t % s.OW);
    long r_ = t / s.OW;
    const int oh = (int)(r_ % s.OH);
    r_ /= s.OH;
    const int cb = (int)(r_ % CB);
    const long n = r_ / CB;
    const int8_t* xb = x + (n * CB + cb) * s.H * s.W * 16;
    const int ih0 = oh * s.sh - s.ph, iw0 = ow * s.sw - s.pw;
    int m[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) m[i] = -128;
    for (int r = 0; r < s.R; ++r) {
        const int ih = ih0 + r;
        if ((unsigned)ih >= (unsigned)s.H) continue;
        for (int c = 0; c < s.S; ++c) {
            const int iw = iw0 + c;
            if ((unsigned)iw >= (unsigned)s.W) continue;
            union {
                int4 v;
                int8_t b[16];
            } u;
            u.v = *reinterpret_cast<const int4*>(xb + ((long)ih * s.W + iw) * 16);
#pragma unroll
            for (int i = 0; i < 16; ++i) m[i] = u.b[i] > m[i] ? u.b[i] : m[i];
        }
    }
    union {
        int4 v;
        int8_t b[16];
    } o;
#pragma unroll
    for (int i = 0; i < 16; ++i) o.b[i] = (int8_t)m[i];
    const int qtot = q.q_tot > 0 ? q.q_tot : CB;
    const long at = (((n * qtot + q.q_off + cb) * (s.OH + 2 * q.qph) + oh + q.qph) * (long)(s.OW + 2 * q.qpw) + ow +
                     q.qpw) * 16;
    *reinterpret_cast<int4*>(q.yq + at) = o.v;
}

hipError_t launch_maxpool_i8(const PoolShape& s, const int8_t* x8, const PoolQ& q, hipStream_t st) {
    const int CB = cdiv(s.C, 16);
    const long total = (long)s.N * CB * s.OH * s.OW;
    if (s.xb != 16 || !x8 || !q.yq || total <= 0 || s.ph >= s.R || s.pw >= s.S) return hipErrorInvalidValue;
    hipLaunchKernelGGL(maxpool_i8_blk, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, x8, s, CB, q);
    return hipGetLastError();
}

hipError_t launch_gap(const float* x, int xb, int N, int C, int H, int W, float* y, hipStream_t st) {
    if (!pow2_block(xb)) return hipErrorInvalidValue;
    const int XB = cdiv(C, xb), G16 = cdiv(XB * xb, 16);
    hipLaunchKernelGGL(gap_blk<false>, dim3(cdiv(N * G16, 4)), dim3(256), 0, st, x, y, N, G16, XB,
                       ilog2(xb), H * W);
    return hipGetLastError();
}

hipError_t launch_gap_q(const float* x, int N, int C, int H, int W, float* y, int8_t* yq, float scale,
                        hipStream_t st) {
    // block 16, C a multiple of 16: the means of image n are the row n * C ...
    if (C % 16 || !x || !yq || !(scale > 0.f)) return hipErrorInvalidValue;
    const int XB = C / 16, G16 = XB;
    hipLaunchKernelGGL(gap_blk<true>, dim3(cdiv(N * G16, 4)), dim3(256), 0, st, x, y, N, G16, XB, 4, H * W, yq,
                       scale, C);
    return hipGetLastError();
}

}  // namespace neo
