// Dense layer y = act(W x + b) on fp32 MFMA, default layout (the operation
// after the layout-dependent Flatten of Section 3.2).
//
// Same 16x16x4 MFMA tiling as the convolution: A = 16 rows of W (output
// features), B = 16 rows of x (batch), D[4g+v][i] = y[batch i][feature 4g+v].
// Both operands are row-major along the reduction axis, so each lane loads one
// float4 per operand per 16-wide reduction chunk.  The chunks are split over
// the 4 waves of a workgroup and summed through LDS in a fixed order.  At batch
// 1 the layer is a weight stream (HBM bound); U chunks of loads are issued
// before their MFMAs to keep enough bytes in flight.
#include "neo_internal.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

struct DenseArgs {
    const float* x;
    const float* w;
    const float* bias;
    float* y;
    int N, IN, OUT, act, T;  // T = number of 16-wide reduction chunks
};

constexpr int kWaves = 4;
constexpr int kU = 4;

// Load 4 consecutive reduction elements starting at k of a row; VEC = row
// starts are 16-byte aligned (IN % 4 == 0), so a chunk is all in or all out.
template <bool VEC>
__device__ inline v4f load4(const float* row, int k, int IN, bool rowok) {
    v4f v = v4f{0.f, 0.f, 0.f, 0.f};
    if (!rowok) return v;
    if constexpr (VEC) {
        if (k < IN) v = *reinterpret_cast<const v4f*>(row + k);
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (k + i < IN) v[i] = row[k + i];
    }
    return v;
}

template <int FO, int FN, bool VEC>
__global__ __launch_bounds__(256) void dense_mfma(DenseArgs a) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;
    const int o0 = blockIdx.x * 16 * FO;
    const int n0 = blockIdx.y * 16 * FN;

    const float* wr[FO];
    bool wok[FO];
#pragma unroll
    for (int f = 0; f < FO; ++f) {
        const int o = o0 + 16 * f + li;
        wok[f] = o < a.OUT;
        wr[f] = a.w + (long)(wok[f] ? o : 0) * a.IN;
    }
    const float* xr[FN];
    bool xok[FN];
#pragma unroll
    for (int p = 0; p < FN; ++p) {
        const int n = n0 + 16 * p + li;
        xok[p] = n < a.N;
        xr[p] = a.x + (long)(xok[p] ? n : 0) * a.IN;
    }

    v4f acc[FO][FN];
#pragma unroll
    for (int f = 0; f < FO; ++f)
#pragma unroll
        for (int p = 0; p < FN; ++p) acc[f][p] = v4f{0.f, 0.f, 0.f, 0.f};

    for (int c0 = wave; c0 < a.T; c0 += kWaves * kU) {
        v4f wa[kU][FO], xb[kU][FN];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int c = c0 + u * kWaves;
            const int k = c * 16 + 4 * g;
            const bool in = c < a.T;
#pragma unroll
            for (int f = 0; f < FO; ++f) wa[u][f] = load4<VEC>(wr[f], k, a.IN, in && wok[f]);
#pragma unroll
            for (int p = 0; p < FN; ++p) xb[u][p] = load4<VEC>(xr[p], k, a.IN, in && xok[p]);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int f = 0; f < FO; ++f)
#pragma unroll
                    for (int p = 0; p < FN; ++p)
                        acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[u][f][t], xb[u][p][t],
                                                                         acc[f][p], 0, 0, 0);
    }

    __shared__ float red[kWaves - 1][FO * FN * 4][64];
    if (wave > 0) {
#pragma unroll
        for (int f = 0; f < FO; ++f)
#pragma unroll
            for (int p = 0; p < FN; ++p)
#pragma unroll
                for (int v = 0; v < 4; ++v) red[wave - 1][(f * FN + p) * 4 + v][lane] = acc[f][p][v];
    }
    __syncthreads();
    if (wave != 0) return;

#pragma unroll
    for (int f = 0; f < FO; ++f) {
#pragma unroll
        for (int p = 0; p < FN; ++p) {
            const int n = n0 + 16 * p + li;
            if (n >= a.N) continue;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int o = o0 + 16 * f + 4 * g + v;
                if (o >= a.OUT) continue;
                const int q = (f * FN + p) * 4 + v;
                float r = ((acc[f][p][v] + red[0][q][lane]) + red[1][q][lane]) + red[2][q][lane];
                if (a.bias) r += a.bias[o];
                if (a.act == NEO_ACT_RELU) r = r > 0.f ? r : 0.f;
                a.y[(long)n * a.OUT + o] = r;
            }
        }
    }
}

template <int FO, int FN, bool VEC>
hipError_t launch_t(const DenseArgs& a, hipStream_t st) {
    dim3 grid(cdiv(a.OUT, 16 * FO), cdiv(a.N, 16 * FN));
    hipLaunchKernelGGL((dense_mfma<FO, FN, VEC>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

template <bool VEC>
hipError_t dispatch(const DenseArgs& a, hipStream_t st) {
    if (a.N <= 16) return launch_t<1, 1, VEC>(a, st);
    return launch_t<1, 2, VEC>(a, st);
}

}  // namespace

hipError_t launch_dense(const float* x, int N, int IN, const float* w, int OUT,
                        const float* bias, int act, float* y, hipStream_t st) {
    DenseArgs a{x, w, bias, y, N, IN, OUT, act, cdiv(IN, 16)};
    const bool vec = (IN % 4 == 0) && aligned16(x) && aligned16(w);
    return vec ? dispatch<true>(a, st) : dispatch<false>(a, st);
}

}  // namespace neo
