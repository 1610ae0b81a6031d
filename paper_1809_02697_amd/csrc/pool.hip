// Layout-tolerant pooling on NCHW16c (Section 3.2): max, average, global
// average.  One thread per (output pixel, 4-channel quad) moves float4s, so a
// wave reads and writes 16 pixels x 64 bytes = 1 KB contiguous per access.
// Max pooling ignores taps outside the input (as if padded with -inf); average
// pooling divides by the number of taps inside it.
// Padded channel lanes hold 0 in the input and stay 0 in the output.
#include "neo_internal.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

// Taps of a KR x KS window (0 = the window from the shape, a runtime loop).
// With a compile-time window every tap's load is issued before any is used:
// a tap outside the input loads pixel (0, 0) of the block and is discarded by
// a select, so the loads of one output are in flight together.
template <bool MAX, int KR, int KS>
__global__ __launch_bounds__(256) void pool_b16(const float* __restrict__ x, float* __restrict__ y,
                                                PoolShape s, int CB) {
    const int total = s.N * CB * s.OH * s.OW * 4;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int q = t & 3;
        int r_ = t >> 2;
        const int ow = r_ % s.OW;
        r_ /= s.OW;
        const int oh = r_ % s.OH;
        r_ /= s.OH;
        const int cb = r_ % CB;
        const int n = r_ / CB;
        const float* xb = x + (n * CB + cb) * s.H * s.W * 16 + 4 * q;
        const int ih0 = oh * s.sh - s.ph, iw0 = ow * s.sw - s.pw;
        v4f acc;
        if (MAX)
            acc = v4f{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        else
            acc = v4f{0.f, 0.f, 0.f, 0.f};
        int cnt = 0;
        if constexpr (KR > 0) {
            v4f v[KR][KS];
            bool ok[KR][KS];
#pragma unroll
            for (int r = 0; r < KR; ++r)
#pragma unroll
                for (int c = 0; c < KS; ++c) {
                    const int ih = ih0 + r, iw = iw0 + c;
                    ok[r][c] = (unsigned)ih < (unsigned)s.H && (unsigned)iw < (unsigned)s.W;
                    v[r][c] = *reinterpret_cast<const v4f*>(xb + (ok[r][c] ? ih * s.W + iw : 0) * 16);
                }
#pragma unroll
            for (int r = 0; r < KR; ++r)
#pragma unroll
                for (int c = 0; c < KS; ++c) {
                    if (!ok[r][c]) continue;
                    if (MAX) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[i] = v[r][c][i] > acc[i] ? v[r][c][i] : acc[i];
                    } else {
                        acc += v[r][c];
                    }
                    ++cnt;
                }
        } else {
            for (int r = 0; r < s.R; ++r) {
                const int ih = ih0 + r;
                if ((unsigned)ih >= (unsigned)s.H) continue;
                for (int c = 0; c < s.S; ++c) {
                    const int iw = iw0 + c;
                    if ((unsigned)iw >= (unsigned)s.W) continue;
                    const v4f v = *reinterpret_cast<const v4f*>(xb + (ih * s.W + iw) * 16);
                    if (MAX) {
#pragma unroll
                        for (int i = 0; i < 4; ++i) acc[i] = v[i] > acc[i] ? v[i] : acc[i];
                    } else {
                        acc += v;
                    }
                    ++cnt;
                }
            }
        }
        if (!MAX) {
            const float d = (float)cnt;
#pragma unroll
            for (int i = 0; i < 4; ++i) acc[i] = acc[i] / d;
        }
        *reinterpret_cast<v4f*>(y + (((n * s.y_tot + s.y_off + cb) * s.OH + oh) * s.OW + ow) * 16 +
                                4 * q) = acc;
    }
}

// One wave per (n, channel block): lane = 4 * pixel_slot + quad; each lane sums
// the pixels p = slot, slot + 16, ... of its quad, then the 16 slots are summed
// with cross-lane shuffles in a fixed tree order.
__global__ __launch_bounds__(256) void gap_b16(const float* __restrict__ x, float* __restrict__ y,
                                               int NCB, int HW) {
    const int wave_id = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (wave_id >= NCB) return;
    const int lane = threadIdx.x & 63;
    const int q = lane & 3, slot = lane >> 2;
    const float* xb = x + wave_id * HW * 16 + 4 * q;
    v4f acc = v4f{0.f, 0.f, 0.f, 0.f};
    int p = slot;
    for (; p + 48 < HW; p += 64) {  // four pixels of the slot in flight
        v4f v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = *reinterpret_cast<const v4f*>(xb + (p + 16 * u) * 16);
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += v[u];
    }
    for (; p < HW; p += 16) acc += *reinterpret_cast<const v4f*>(xb + p * 16);
#pragma unroll
    for (int off = 4; off < 64; off <<= 1) {
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] += __shfl_xor(acc[i], off, 64);
    }
    if (slot == 0) {
        const float d = (float)HW;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = acc[i] / d;
        *reinterpret_cast<v4f*>(y + wave_id * 16 + 4 * q) = acc;
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
    const int CB = cdiv(s.C, 16);
    const dim3 g = grid_for((long)s.N * CB * s.OH * s.OW * 4), b(256);
    if (s.R == 3 && s.S == 3)
        hipLaunchKernelGGL((pool_b16<MAX, 3, 3>), g, b, 0, st, x, y, s, CB);
    else if (s.R == 2 && s.S == 2)
        hipLaunchKernelGGL((pool_b16<MAX, 2, 2>), g, b, 0, st, x, y, s, CB);
    else
        hipLaunchKernelGGL((pool_b16<MAX, 0, 0>), g, b, 0, st, x, y, s, CB);
    return hipGetLastError();
}

hipError_t launch_maxpool(const PoolShape& s, const float* x, float* y, hipStream_t st) {
    return launch_pool<true>(s, x, y, st);
}

hipError_t launch_avgpool(const PoolShape& s, const float* x, float* y, hipStream_t st) {
    return launch_pool<false>(s, x, y, st);
}

hipError_t launch_gap(const float* x, int N, int C, int H, int W, float* y, hipStream_t st) {
    const int NCB = N * cdiv(C, 16);
    hipLaunchKernelGGL(gap_b16, dim3(cdiv(NCB, 4)), dim3(256), 0, st, x, y, NCB, H * W);
    return hipGetLastError();
}

}  // namespace neo
