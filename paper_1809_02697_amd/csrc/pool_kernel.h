// Max and average pooling of one output quad on NCHW[x]c (Section 3.2: a
// layout-tolerant operation), shared by the pooling kernel and by fused conv
// launches that run a pooling step in their last workgroups, so both compute
// the same bits.
#pragma once

#include <cmath>

#include "neo_internal.h"

namespace neo {
namespace pool_detail {

typedef float v4f __attribute__((ext_vector_type(4)));

// Thread index t = (((n * CB + cb) * OH + oh) * OW + ow) * (x / 4) + quad, for
// t < (N * CB * OH * OW) << lq (lq = log2(x / 4)).  Taps outside the input are
// skipped (max: as if padded with -inf; average: divided by the taps inside).
// The average sums in double, row by row, and rounds once to float32 after
// the division: the result is the exact mean rounded, whatever the hardware
// (the float32 sum of the same taps could differ in its last bit).
// With a compile-time KR x KS window every tap's load is issued before any is
// used: a tap outside the input loads pixel (0, 0) of the block and is
// discarded by a select, so the loads of one output are in flight together;
// KR = 0 walks the window from the shape.  Both walk the taps row by row, so
// the sums are the same.
// Q: the output may also (or only: y null) be written as its int8 copy q
// (block 16, one quad of four channels = four bytes of the pixel's 16).
template <bool MAX, int KR, int KS, bool Q = false>
__device__ __forceinline__ void pool_elem(const float* __restrict__ x, float* __restrict__ y,
                                          const PoolShape& s, int CB, int lq, int t,
                                          const PoolQ& q = PoolQ{}) {
    const int X = s.xb;
    const int qd = t & ((1 << lq) - 1);
    int r_ = t >> lq;
    const int ow = r_ % s.OW;
    r_ /= s.OW;
    const int oh = r_ % s.OH;
    r_ /= s.OH;
    const int cb = r_ % CB;
    const int n = r_ / CB;
    const float* xb = x + (n * CB + cb) * s.H * s.W * X + 4 * qd;
    const int ih0 = oh * s.sh - s.ph, iw0 = ow * s.sw - s.pw;
    v4f acc;
    if (MAX)
        acc = v4f{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    else
        acc = v4f{0.f, 0.f, 0.f, 0.f};
    double dacc[4] = {0.0, 0.0, 0.0, 0.0};
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
                v[r][c] = *reinterpret_cast<const v4f*>(xb + (ok[r][c] ? ih * s.W + iw : 0) * X);
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
#pragma unroll
                    for (int i = 0; i < 4; ++i) dacc[i] += (double)v[r][c][i];
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
                const v4f v = *reinterpret_cast<const v4f*>(xb + (ih * s.W + iw) * X);
                if (MAX) {
#pragma unroll
                    for (int i = 0; i < 4; ++i) acc[i] = v[i] > acc[i] ? v[i] : acc[i];
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i) dacc[i] += (double)v[i];
                }
                ++cnt;
            }
        }
    }
    if (!MAX) {
        const double d = (double)cnt;
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[i] = (float)(dacc[i] / d);
    }
    if (!Q || y) *reinterpret_cast<v4f*>(y + (((n * s.y_tot + s.y_off + cb) * s.OH + oh) * s.OW + ow) * X + 4 * qd) = acc;
    if constexpr (Q) {
        if (q.yq) {
            // clamp(round_half_even(v / scale), -127, 127), the division in float32
            unsigned packed = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float r = rintf(acc[i] / q.scale);
                r = r > 127.f ? 127.f : (r < -127.f ? -127.f : r);
                packed |= ((unsigned)(int)r & 0xffu) << (8 * i);
            }
            const int owq = s.OW + 2 * q.qpw;
            const int qtot = q.q_tot > 0 ? q.q_tot : CB;
            const long at =
                (((long)(n * qtot + q.q_off + cb) * (s.OH + 2 * q.qph) + oh + q.qph) * owq + ow + q.qpw) * 16 + 4 * qd;
            *reinterpret_cast<unsigned*>(q.yq + at) = packed;
        }
    }
}

}  // namespace pool_detail
}  // namespace neo
