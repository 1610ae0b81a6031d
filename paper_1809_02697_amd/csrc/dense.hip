// Dense layer y = act(W x + b) on fp32 MFMA, default layout (the operation
// after the layout-dependent Flatten of Section 3.2).
//
// Same 16x16x4 MFMA tiling as the convolution: A = 16 rows of W (output
// features), B = 16 rows of x (batch), D[4g+v][i] = y[batch i][feature 4g+v].
// Both operands are row-major along the reduction axis, so each lane loads one
// float4 per operand per 16-wide reduction chunk.  The chunks are split over
// the 4 waves of a workgroup and summed through LDS in a fixed order; U chunks
// of loads are issued before their MFMAs to keep enough bytes in flight.
//
// Up to 4 batch rows the layer is a matrix-vector product, a pure weight
// stream (HBM bound), and a 16-wide MFMA tile would waste 15/16 of its batch
// lanes while giving too few workgroups to keep HBM busy.  That case runs
// dense_rows: one wave per output feature, so the grid has OUT/4 workgroups
// and every lane keeps G float4 loads of its row in flight.
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
    // x is the mean of `parts` rows (stride xs4 float4s): scale * (row 0 + row 1 + ...)
    int parts, xs4;
    float scale;
};

// float4 k of the mean of the input's rows (in row order)
__device__ inline v4f rows_mean4(const DenseArgs& a, const v4f* x4, int k) {
    v4f s = x4[k];
    for (int t = 1; t < a.parts; ++t) s += x4[(long)t * a.xs4 + k];
    return s * a.scale;
}

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

constexpr int kG = 8;  // float4 chunks of a row in flight per lane
constexpr int kMaxPartsIn = 16384;  // an input summed into LDS: at most 64 KB

// One wave per output feature o: lane l accumulates the chunks l, l+64, ...
// of row o against the same chunks of each batch row, then the wave adds its
// lanes in a fixed butterfly order.  NB >= N batch rows, compile-time.
// PARTS (one batch row): the workgroup first sums the input's rows into LDS
// once, and its waves read the input from there.
template <int NB, bool VEC, bool PARTS = false>
__global__ __launch_bounds__(256) void dense_rows(DenseArgs a) {
    extern __shared__ v4f xsum[];  // PARTS: IN / 4 float4s
    if constexpr (PARTS) {
        const int n4 = a.IN >> 2;
        const v4f* x4 = reinterpret_cast<const v4f*>(a.x);
        for (int k = threadIdx.x; k < n4; k += blockDim.x) xsum[k] = rows_mean4(a, x4, k);
        __syncthreads();
    }
    const int lane = threadIdx.x & 63;
    const int o = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (o >= a.OUT) return;  // whole wave
    const float* wr = a.w + (long)o * a.IN;
    float acc[NB];
#pragma unroll
    for (int n = 0; n < NB; ++n) acc[n] = 0.f;
    if constexpr (VEC) {
        const int n4 = a.IN >> 2;
        const v4f* w4 = reinterpret_cast<const v4f*>(wr);
        const v4f* x4 = reinterpret_cast<const v4f*>(a.x);
        int k = lane;
        for (; k + 64 * (kG - 1) < n4; k += 64 * kG) {
            v4f wv[kG], xv[kG][NB];
#pragma unroll
            for (int g = 0; g < kG; ++g) wv[g] = w4[k + 64 * g];
#pragma unroll
            for (int g = 0; g < kG; ++g)
#pragma unroll
                for (int n = 0; n < NB; ++n) {
                    if constexpr (PARTS)
                        xv[g][n] = xsum[k + 64 * g];
                    else
                        xv[g][n] = n < a.N ? x4[(long)n * n4 + k + 64 * g] : v4f{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll
            for (int g = 0; g < kG; ++g)
#pragma unroll
                for (int n = 0; n < NB; ++n)
                    acc[n] += wv[g].x * xv[g][n].x + wv[g].y * xv[g][n].y + wv[g].z * xv[g][n].z +
                              wv[g].w * xv[g][n].w;
        }
        for (; k < n4; k += 64) {
            const v4f wv = w4[k];
#pragma unroll
            for (int n = 0; n < NB; ++n) {
                if (n >= a.N) break;
                const v4f xv = PARTS ? xsum[k] : x4[(long)n * n4 + k];
                acc[n] += wv.x * xv.x + wv.y * xv.y + wv.z * xv.z + wv.w * xv.w;
            }
        }
    } else {
        static_assert(!PARTS, "partial rows need aligned float4 rows");
        for (int k = lane; k < a.IN; k += 64) {
            const float wv = wr[k];
#pragma unroll
            for (int n = 0; n < NB; ++n)
                if (n < a.N) acc[n] += wv * a.x[(long)n * a.IN + k];
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1)
#pragma unroll
        for (int n = 0; n < NB; ++n) acc[n] += __shfl_xor(acc[n], off, 64);
    if (lane != 0) return;
    const float b = a.bias ? a.bias[o] : 0.f;
#pragma unroll
    for (int n = 0; n < NB; ++n) {
        if (n >= a.N) break;
        float r = acc[n] + b;
        if (a.act == NEO_ACT_RELU) r = r > 0.f ? r : 0.f;
        a.y[(long)n * a.OUT + o] = r;
    }
}

template <int NB, bool VEC>
hipError_t launch_rows(const DenseArgs& a, hipStream_t st) {
    hipLaunchKernelGGL((dense_rows<NB, VEC>), dim3(cdiv(a.OUT, 4)), dim3(256), 0, st, a);
    return hipGetLastError();
}

template <int FO, int FN, bool VEC>
hipError_t launch_t(const DenseArgs& a, hipStream_t st) {
    dim3 grid(cdiv(a.OUT, 16 * FO), cdiv(a.N, 16 * FN));
    hipLaunchKernelGGL((dense_mfma<FO, FN, VEC>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

template <bool VEC>
hipError_t dispatch(const DenseArgs& a, hipStream_t st) {
    if (a.N == 1) return launch_rows<1, VEC>(a, st);
    if (a.N == 2) return launch_rows<2, VEC>(a, st);
    if (a.N <= 4) return launch_rows<4, VEC>(a, st);
    if (a.N <= 16) return launch_t<1, 1, VEC>(a, st);
    return launch_t<1, 2, VEC>(a, st);
}

}  // namespace

hipError_t launch_dense_parts(const float* x, int parts, int xstride, float scale, int IN,
                              const float* w, int OUT, const float* bias, int act, float* y,
                              hipStream_t st) {
    if (parts < 1 || xstride < IN || xstride % 4 || IN % 4 || IN > kMaxPartsIn || !aligned16(x) ||
        !aligned16(w))
        return hipErrorInvalidValue;
    DenseArgs a{x, w, bias, y, 1, IN, OUT, act, cdiv(IN, 16), parts, xstride / 4, scale};
    hipLaunchKernelGGL((dense_rows<1, true, true>), dim3(cdiv(OUT, 4)), dim3(256), IN * 4, st, a);
    return hipGetLastError();
}

hipError_t launch_dense(const float* x, int N, int IN, const float* w, int OUT,
                        const float* bias, int act, float* y, hipStream_t st) {
    DenseArgs a{x, w, bias, y, N, IN, OUT, act, cdiv(IN, 16), 0, 0, 1.f};
    const bool vec = (IN % 4 == 0) && aligned16(x) && aligned16(w);
    return vec ? dispatch<true>(a, st) : dispatch<false>(a, st);
}

}  // namespace neo
