// Blocked convolution on fp32 MFMA (gfx950).
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
// channels of a block is free).  Filter loads: the KCRS[16]c[16]k block of one
// (kb, cb, r, s) is [16 c][16 k]; the lane reads w[c = 4g+t][k = i], 16
// consecutive floats per c row.
//
// The reduction steps of a workgroup's output tile are split over its 4 waves
// (step st goes to wave st % 4) and summed through LDS in a fixed order, so the
// result is deterministic.  The epilogue (bias, residual, ReLU) runs in
// registers before the single store.
#include "neo_internal.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

struct ConvArgs {
    const float* x;
    const float* w;
    const float* bias;
    const float* res;
    float* y;
    int N, CB, H, W, KB, R, S, RS, sh, sw, ph, pw, OH, OW, M, y_off, y_tot, act, T;
};

constexpr int kWaves = 4;

template <int FK, int FP, bool SMALLC>
__global__ __launch_bounds__(256) void conv2d_mfma(ConvArgs a) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int li = lane & 15;
    const int g = lane >> 4;
    const int m0 = blockIdx.x * (16 * FP);
    const int kb0 = blockIdx.y * FK;
    const int ohw = a.OH * a.OW;

    int pn[FP], poh[FP], pow_[FP];
    bool pv[FP];
#pragma unroll
    for (int p = 0; p < FP; ++p) {
        const int m = m0 + 16 * p + li;
        pv[p] = m < a.M;
        const int mm = pv[p] ? m : 0;
        const int n = mm / ohw;
        const int rem = mm - n * ohw;
        const int oh = rem / a.OW;
        pn[p] = n;
        poh[p] = oh;
        pow_[p] = rem - oh * a.OW;
    }

    v4f acc[FK][FP];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int p = 0; p < FP; ++p) acc[f][p] = v4f{0.f, 0.f, 0.f, 0.f};

    for (int st = wave; st < a.T; st += kWaves) {
        const int cb = st / a.RS;
        const int rs = st - cb * a.RS;
        const int r = rs / a.S;
        const int s = rs - r * a.S;
        if constexpr (!SMALLC) {
            v4f b[FP];
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                const int ih = poh[p] * a.sh - a.ph + r;
                const int iw = pow_[p] * a.sw - a.pw + s;
                const bool ok = pv[p] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                b[p] = v4f{0.f, 0.f, 0.f, 0.f};
                if (ok)
                    b[p] = *reinterpret_cast<const v4f*>(
                        a.x + (((pn[p] * a.CB + cb) * a.H + ih) * a.W + iw) * 16 + 4 * g);
            }
            float wa[FK][4];
#pragma unroll
            for (int f = 0; f < FK; ++f) {
                const int kb = kb0 + f;
                if (kb < a.KB) {
                    const float* wp = a.w + ((kb * a.CB + cb) * a.RS + rs) * 256 + (4 * g) * 16 + li;
#pragma unroll
                    for (int t = 0; t < 4; ++t) wa[f][t] = wp[16 * t];
                } else {
#pragma unroll
                    for (int t = 0; t < 4; ++t) wa[f][t] = 0.f;
                }
            }
#pragma unroll
            for (int t = 0; t < 4; ++t)
#pragma unroll
                for (int f = 0; f < FK; ++f)
#pragma unroll
                    for (int p = 0; p < FP; ++p)
                        acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[f][t], b[p][t],
                                                                         acc[f][p], 0, 0, 0);
        } else {
            // At most 4 real input channels (one block, cb = 0): lane group g
            // carries input channel g, so each kernel entry is one k-step and
            // the 12 zero-padded channels are never multiplied.
            float b[FP];
#pragma unroll
            for (int p = 0; p < FP; ++p) {
                const int ih = poh[p] * a.sh - a.ph + r;
                const int iw = pow_[p] * a.sw - a.pw + s;
                const bool ok = pv[p] && (unsigned)ih < (unsigned)a.H && (unsigned)iw < (unsigned)a.W;
                b[p] = ok ? a.x[((pn[p] * a.CB) * a.H + ih) * a.W * 16 + iw * 16 + g] : 0.f;
            }
#pragma unroll
            for (int f = 0; f < FK; ++f) {
                const int kb = kb0 + f;
                const float wv = kb < a.KB ? a.w[(kb * a.CB * a.RS + rs) * 256 + g * 16 + li] : 0.f;
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(wv, b[p], acc[f][p], 0, 0, 0);
            }
        }
    }

    // Sum the four waves' partial tiles (fixed order: wave 0 + 1 + 2 + 3).
    __shared__ float red[kWaves - 1][FK * FP * 4][64];
    if (wave > 0) {
#pragma unroll
        for (int f = 0; f < FK; ++f)
#pragma unroll
            for (int p = 0; p < FP; ++p)
#pragma unroll
                for (int v = 0; v < 4; ++v) red[wave - 1][(f * FP + p) * 4 + v][lane] = acc[f][p][v];
    }
    __syncthreads();
    if (wave != 0) return;

#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kb0 + f;
        if (kb >= a.KB) continue;
        v4f bb = v4f{0.f, 0.f, 0.f, 0.f};
        if (a.bias) bb = *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * g);
#pragma unroll
        for (int p = 0; p < FP; ++p) {
            if (!pv[p]) continue;
            v4f o = acc[f][p];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int q = (f * FP + p) * 4 + v;
                o[v] = ((o[v] + red[0][q][lane]) + red[1][q][lane]) + red[2][q][lane];
            }
            o += bb;
            if (a.res) {
                const v4f rv = *reinterpret_cast<const v4f*>(
                    a.res + (((pn[p] * a.KB + kb) * a.OH + poh[p]) * a.OW + pow_[p]) * 16 + 4 * g);
                o += rv;
            }
            if (a.act == NEO_ACT_RELU) {
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
            }
            *reinterpret_cast<v4f*>(
                a.y + (((pn[p] * a.y_tot + a.y_off + kb) * a.OH + poh[p]) * a.OW + pow_[p]) * 16 +
                4 * g) = o;
        }
    }
}

template <int FK, int FP, bool SMALLC>
hipError_t launch_t(const ConvArgs& a, hipStream_t st) {
    dim3 grid(cdiv(a.M, 16 * FP), cdiv(a.KB, FK));
    hipLaunchKernelGGL((conv2d_mfma<FK, FP, SMALLC>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

template <bool SMALLC>
hipError_t dispatch(int fk, int fp, const ConvArgs& a, hipStream_t st) {
    switch (fk * 8 + fp) {
        case 1 * 8 + 1: return launch_t<1, 1, SMALLC>(a, st);
        case 1 * 8 + 2: return launch_t<1, 2, SMALLC>(a, st);
        case 1 * 8 + 4: return launch_t<1, 4, SMALLC>(a, st);
        case 2 * 8 + 1: return launch_t<2, 1, SMALLC>(a, st);
        case 2 * 8 + 2: return launch_t<2, 2, SMALLC>(a, st);
        case 2 * 8 + 4: return launch_t<2, 4, SMALLC>(a, st);
        case 4 * 8 + 1: return launch_t<4, 1, SMALLC>(a, st);
        case 4 * 8 + 2: return launch_t<4, 2, SMALLC>(a, st);
        case 4 * 8 + 4: return launch_t<4, 4, SMALLC>(a, st);
        default: return hipErrorInvalidValue;
    }
}

// Largest register tile that still gives every CU at least one workgroup.
void pick_tile(int M, int KB, int* fk, int* fp) {
    static const int cand[][2] = {{4, 4}, {4, 2}, {2, 4}, {2, 2}, {4, 1}, {1, 4},
                                  {2, 1}, {1, 2}, {1, 1}};
    const int MP = cdiv(M, 16);
    for (const auto& c : cand) {
        if (c[0] > KB && KB >= 1 && c[0] > 1) continue;
        if ((long)cdiv(MP, c[1]) * cdiv(KB, c[0]) >= 256) {
            *fk = c[0];
            *fp = c[1];
            return;
        }
    }
    *fk = 1;
    *fp = 1;
}

}  // namespace

hipError_t launch_conv2d(const ConvShape& s, const float* x, const float* w, const float* bias,
                         const float* res, float* y, hipStream_t st) {
    ConvArgs a;
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.res = res;
    a.y = y;
    a.N = s.N;
    a.CB = cdiv(s.C, 16);
    a.H = s.H;
    a.W = s.W;
    a.KB = cdiv(s.K, 16);
    a.R = s.R;
    a.S = s.S;
    a.RS = s.R * s.S;
    a.sh = s.sh;
    a.sw = s.sw;
    a.ph = s.ph;
    a.pw = s.pw;
    a.OH = s.OH;
    a.OW = s.OW;
    a.M = s.N * s.OH * s.OW;
    a.y_off = s.y_off;
    a.y_tot = s.y_tot;
    a.act = s.act;
    a.T = a.CB * a.RS;
    int fk, fp;
    pick_tile(a.M, a.KB, &fk, &fp);
    if (s.C <= 4) return dispatch<true>(fk, fp, a, st);
    return dispatch<false>(fk, fp, a, st);
}

}  // namespace neo
