// Winograd minimal filtering F(2x2, 3x3): the filter transform, shared by the
// host (plans) and the device (the standalone filter call), so both produce
// the same bits.
//
// F(m, r) computes m outputs of an r-tap correlation from m + r - 1 inputs
// with m + r - 1 multiplications (Winograd's minimal filtering algorithm, as
// applied to convolutional layers by Lavin and Gray, "Fast Algorithms for
// Convolutional Neural Networks", 2016).  Nested in two dimensions, a 2x2
// output tile of a 3x3 correlation is
//   Y = A^T [ (G g G^T) .* (B^T d B) ] A
// over the tile's 4x4 input patch d, with
//   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1],
//   G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1],
//   A^T = [1 1 1 0; 0 1 -1 -1].
// The element-wise product, summed over input channels, is 16 independent
// matrix products (one per element of the 4x4 transformed tile) -- the part
// that runs on MFMA.  The halves sit in the filter transform, so the input and
// output transforms are additions only.
#pragma once

#include <hip/hip_runtime.h>

namespace neo {

// Element block of the transformed filter: for output block kb, input block
// cb and element e = 4 i + j of the 4x4 transformed tile, 256 floats in the
// MFMA operand order [c/4][k][c%4] (lane (k, g) reads channels 4g..4g+3 of
// output channel k as one float4).  Blocks are stored [kb][cb][e].
constexpr int kWinoElems = 16;

__host__ __device__ inline long wino_filter_index(int CB, int k, int c, int e) {
    const int kb = k >> 4, kk = k & 15, cb = c >> 4, cc = c & 15;
    return (((long)kb * CB + cb) * kWinoElems + e) * 256 + ((cc >> 2) * 16 + kk) * 4 + (cc & 3);
}

// G applied to three taps: (t0, (t0 + t1 + t2) / 2, (t0 - t1 + t2) / 2, t2).
// Halving is exact, and there is no product to contract into a fused
// multiply-add, so host and device round identically.
__host__ __device__ inline void wino_g(double t0, double t1, double t2, double* o) {
    o[0] = t0;
    o[1] = (t0 + t1 + t2) * 0.5;
    o[2] = (t0 - t1 + t2) * 0.5;
    o[3] = t2;
}

// U = G g G^T of one 3x3 filter g[r][s] (row-major), in double, each element
// rounded once to float: u[4 i + j].
__host__ __device__ inline void wino_filter_tile(const float* g, float* u) {
    double gc[4][3];  // G g: columns s of g transformed
    for (int s = 0; s < 3; ++s) {
        double o[4];
        wino_g(g[s], g[3 + s], g[6 + s], o);
        for (int i = 0; i < 4; ++i) gc[i][s] = o[i];
    }
    for (int i = 0; i < 4; ++i) {
        double o[4];
        wino_g(gc[i][0], gc[i][1], gc[i][2], o);
        for (int j = 0; j < 4; ++j) u[4 * i + j] = (float)o[j];
    }
}

}  // namespace neo
