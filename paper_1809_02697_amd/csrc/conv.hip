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
// Work split.  Algorithm 1 parallelizes over disjoint output chunks only; at
// batch 1 that leaves too few chunks for 1024 SIMDs, so the reduction is split
// as well:
//   - across the 4 waves of a workgroup (step st goes to wave st % 4), summed
//     through LDS in wave order;
//   - across SPLIT workgroups (grid z), each owning a contiguous range of
//     steps.  Every workgroup writes its partial tile to a workspace and bumps
//     a per-tile counter; the workgroup that arrives last sums the SPLIT
//     partials in split order (so the result does not depend on arrival
//     order), resets the counter to 0 for the next launch and runs the
//     epilogue.  No workgroup ever waits for another.
// Loads run D steps ahead of the MFMAs (a register ring sized to the tile), so
// each wave keeps D-1 steps of loads in flight while it computes.
// The epilogue (bias, residual, ReLU) runs in registers before the single store.
#include <algorithm>
#include <cmath>

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
    float* ws;     // split partials [SPLIT][tiles][FK*FP][64 lanes][4]
    int* cnt;      // per-tile arrival counters (0 between launches)
    int N, CB, H, W, KB, R, S, RS, sh, sw, ph, pw, OH, OW, M, y_off, y_tot, act, T, split;
};

constexpr int kWaves = 4;

template <int FK, int FP, bool SMALLC>
struct Operands;

template <int FK, int FP>
struct Operands<FK, FP, false> {
    v4f b[FP];
    float a[FK][4];
};

template <int FK, int FP>
struct Operands<FK, FP, true> {
    float b[FP];
    float a[FK];
};

// One reduction step (channel block cb, kernel entry r, s): the input offset
// relative to the pixel's own address, (cb*H*W + r*W + s)*16 floats, and the
// tap (r, s) for the zero-padding test.  Built once per workgroup in LDS so
// the inner loop never divides.
struct StepInfo {
    int dx;
    short r, s;
};

constexpr int kMaxTableSteps = 2048;

template <int FK, int FP, bool SMALLC, bool PW>
struct Tile {
    // per-lane pixel coordinates of the FP pixel groups (lanes past the last
    // pixel are clamped to pixel 0: their results are never stored)
    int pbase[FP], pih[FP], piw[FP];
    const float* wbase[FK];  // channel blocks past K are clamped to block 0

    // Every load is issued unconditionally (zero-padding taps read a clamped
    // address and are zeroed by a select) so the number of loads in flight
    // is static and the compiler waits only for the step it is about to use.
    // PW: 1x1 window, no padding: every tap is in bounds and step st is
    // channel block st.
    __device__ void load(const ConvArgs& a, const StepInfo (&tab)[PW ? 1 : kMaxTableSteps],
                         bool use_tab, int k_lo, int st, int g, int li,
                         Operands<FK, FP, SMALLC>& o) const {
        int dx, r = 0, s = 0;
        if constexpr (PW) {
            dx = st * a.H * a.W * 16;
        } else if (use_tab) {
            const StepInfo e = tab[st - k_lo];
            dx = e.dx;
            r = e.r;
            s = e.s;
        } else {
            // range longer than the table: decode (uniform, slower)
            const int cb = st / a.RS;
            const int rs = st - cb * a.RS;
            r = rs / a.S;
            s = rs - r * a.S;
            dx = ((cb * a.H + r) * a.W + s) * 16;
        }
#pragma unroll
        for (int p = 0; p < FP; ++p) {
            bool ok = true;
            if constexpr (!PW) {
                ok = (unsigned)(pih[p] + r) < (unsigned)a.H && (unsigned)(piw[p] + s) < (unsigned)a.W;
            }
            const float* src = a.x + (ok ? pbase[p] + dx : 0);
            if constexpr (!SMALLC) {
                const v4f v = *reinterpret_cast<const v4f*>(src + 4 * g);
#pragma unroll
                for (int i = 0; i < 4; ++i) o.b[p][i] = ok ? v[i] : 0.f;
            } else {
                const float v = src[g];
                o.b[p] = ok ? v : 0.f;
            }
        }
#pragma unroll
        for (int f = 0; f < FK; ++f) {
            const float* wp = wbase[f] + st * 256;
            if constexpr (!SMALLC) {
#pragma unroll
                for (int t = 0; t < 4; ++t) o.a[f][t] = wp[(4 * g + t) * 16 + li];
            } else {
                o.a[f] = wp[g * 16 + li];
            }
        }
    }
};

// Depth of the load ring: as many steps in flight as about 72 VGPRs allow.
template <int FK, int FP, bool SMALLC>
constexpr int pipe_depth() {
    const int regs = SMALLC ? (FK + FP) : 4 * (FK + FP);
    const int d = 72 / regs;
    return d < 2 ? 2 : (d > 8 ? 8 : d);
}

template <int FK, int FP, bool SMALLC>
__device__ inline void mma(const Operands<FK, FP, SMALLC>& o, v4f (&acc)[FK][FP]) {
    if constexpr (!SMALLC) {
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[f][t], o.b[p][t], acc[f][p],
                                                                     0, 0, 0);
    } else {
#pragma unroll
        for (int f = 0; f < FK; ++f)
#pragma unroll
            for (int p = 0; p < FP; ++p)
                acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(o.a[f], o.b[p], acc[f][p], 0, 0, 0);
    }
}

template <int FK, int FP, bool SMALLC, bool PW>
__global__ __launch_bounds__(256) void conv2d_mfma(ConvArgs a) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int li = lane & 15;
    const int g = lane >> 4;
    const int m0 = blockIdx.x * (16 * FP);
    const int kb0 = blockIdx.y * FK;
    const int ohw = a.OH * a.OW;

    Tile<FK, FP, SMALLC, PW> tl;
    bool pv[FP];
    int pn[FP];
#pragma unroll
    for (int p = 0; p < FP; ++p) {
        const int m = m0 + 16 * p + li;
        pv[p] = m < a.M;
        const int mm = pv[p] ? m : 0;
        const int n = mm / ohw;
        const int rem = mm - n * ohw;
        const int oh = rem / a.OW;
        pn[p] = n;
        tl.pih[p] = oh * a.sh - a.ph;
        tl.piw[p] = (rem - oh * a.OW) * a.sw - a.pw;
        // address of (cb = 0, r = 0, s = 0) for this pixel; may lie outside the
        // tensor when the tap is padding (then it is never dereferenced)
        tl.pbase[p] = ((n * a.CB * a.H + tl.pih[p]) * a.W + tl.piw[p]) * 16;
    }
#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kb0 + f;
        tl.wbase[f] = a.w + (kb < a.KB ? kb : 0) * a.CB * a.RS * 256;
    }

    v4f acc[FK][FP];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int p = 0; p < FP; ++p) acc[f][p] = v4f{0.f, 0.f, 0.f, 0.f};

    // this workgroup's contiguous range of reduction steps; this wave takes
    // every 4th of them
    const int z = blockIdx.z;
    const int k_lo = (int)(((long)a.T * z) / a.split);
    const int k_hi = (int)(((long)a.T * (z + 1)) / a.split);
    const int first = k_lo + wave;
    const int nj = first < k_hi ? (k_hi - first + kWaves - 1) / kWaves : 0;

    __shared__ StepInfo tab[PW ? 1 : kMaxTableSteps];
    const bool use_tab = !PW && k_hi - k_lo <= kMaxTableSteps;
    if (use_tab) {
        for (int i = threadIdx.x; i < k_hi - k_lo; i += blockDim.x) {
            const int st = k_lo + i;
            const int cb = st / a.RS;
            const int rs = st - cb * a.RS;
            const int r = rs / a.S;
            const int sx = rs - r * a.S;
            tab[i] = StepInfo{((cb * a.H + r) * a.W + sx) * 16, (short)r, (short)sx};
        }
        __syncthreads();
    }

    if (nj > 0) {
        constexpr int D = pipe_depth<FK, FP, SMALLC>();
        const int last = first + kWaves * (nj - 1);
        Operands<FK, FP, SMALLC> buf[D];
#pragma unroll
        for (int i = 0; i < D - 1; ++i) tl.load(a, tab, use_tab, k_lo, min(first + kWaves * i, last), g, li, buf[i]);
        for (int j0 = 0; j0 < nj; j0 += D) {
#pragma unroll
            for (int u = 0; u < D; ++u) {
                const int j = j0 + u;
                // refill the slot consumed one step ago with step j + D - 1
                // (past the end: the last step again, never used)
                tl.load(a, tab, use_tab, k_lo, min(first + kWaves * (j + D - 1), last), g, li,
                        buf[(u + D - 1) % D]);
                if (j < nj) mma<FK, FP, SMALLC>(buf[u], acc);
            }
        }
    }

    // Sum the four waves' partial tiles (fixed order: wave 0 + 1 + 2 + 3).
    __shared__ v4f red[kWaves - 1][FK * FP][64];
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
            const int q = f * FP + p;
            acc[f][p] = ((acc[f][p] + red[0][q][lane]) + red[1][q][lane]) + red[2][q][lane];
        }

    if (a.split > 1) {
        const int tiles = gridDim.x * gridDim.y;
        const int tile = blockIdx.y * gridDim.x + blockIdx.x;
        v4f* part = reinterpret_cast<v4f*>(a.ws);
#pragma unroll
        for (int q = 0; q < FK * FP; ++q)
            part[((z * tiles + tile) * FK * FP + q) * 64 + lane] = acc[q / FP][q % FP];
        __threadfence();
        int old = 0;
        if (lane == 0) old = atomicAdd(a.cnt + tile, 1);
        old = __shfl(old, 0, 64);
        if (old != a.split - 1) return;
        __threadfence();
#pragma unroll
        for (int q = 0; q < FK * FP; ++q) {
            v4f s = part[(tile * FK * FP + q) * 64 + lane];
            for (int zz = 1; zz < a.split; ++zz) s += part[((zz * tiles + tile) * FK * FP + q) * 64 + lane];
            acc[q / FP][q % FP] = s;
        }
        if (lane == 0) atomicExch(a.cnt + tile, 0);
    }

#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kb0 + f;
        if (kb >= a.KB) continue;
        v4f bb = v4f{0.f, 0.f, 0.f, 0.f};
        if (a.bias) bb = *reinterpret_cast<const v4f*>(a.bias + kb * 16 + 4 * g);
#pragma unroll
        for (int p = 0; p < FP; ++p) {
            if (!pv[p]) continue;
            const int n = pn[p];
            const int oh = (tl.pih[p] + a.ph) / a.sh;
            const int ow = (tl.piw[p] + a.pw) / a.sw;
            v4f o = acc[f][p] + bb;
            if (a.res) {
                o += *reinterpret_cast<const v4f*>(
                    a.res + (((n * a.KB + kb) * a.OH + oh) * a.OW + ow) * 16 + 4 * g);
            }
            if (a.act == NEO_ACT_RELU) {
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
            }
            *reinterpret_cast<v4f*>(
                a.y + (((n * a.y_tot + a.y_off + kb) * a.OH + oh) * a.OW + ow) * 16 + 4 * g) = o;
        }
    }
}

template <int FK, int FP, bool SMALLC, bool PW>
hipError_t launch_t(const ConvArgs& a, hipStream_t st) {
    dim3 grid(cdiv(a.M, 16 * FP), cdiv(a.KB, FK), a.split);
    hipLaunchKernelGGL((conv2d_mfma<FK, FP, SMALLC, PW>), grid, dim3(256), 0, st, a);
    return hipGetLastError();
}

template <bool SMALLC, bool PW>
hipError_t dispatch(int fk, int fp, const ConvArgs& a, hipStream_t st) {
    switch (fk * 8 + fp) {
        case 1 * 8 + 1: return launch_t<1, 1, SMALLC, PW>(a, st);
        case 1 * 8 + 2: return launch_t<1, 2, SMALLC, PW>(a, st);
        case 1 * 8 + 4: return launch_t<1, 4, SMALLC, PW>(a, st);
        case 2 * 8 + 1: return launch_t<2, 1, SMALLC, PW>(a, st);
        case 2 * 8 + 2: return launch_t<2, 2, SMALLC, PW>(a, st);
        case 2 * 8 + 4: return launch_t<2, 4, SMALLC, PW>(a, st);
        case 4 * 8 + 1: return launch_t<4, 1, SMALLC, PW>(a, st);
        case 4 * 8 + 2: return launch_t<4, 2, SMALLC, PW>(a, st);
        case 4 * 8 + 4: return launch_t<4, 4, SMALLC, PW>(a, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

// Cost model for the launch configuration (FK, FP, SPLIT) of one shape.
// Per SIMD: the MFMA cycles it must issue (padded tiles included) and the
// serial chain of one wave (steps x (MFMA cycles + exposed load latency));
// waves resident on a SIMD overlap each other's latency.  A split adds the
// partial round trip through L2 and the last-arrival pass.
ConvConfig choose_conv_config(const ConvShape& s) {
    const int KB = cdiv(s.K, 16), MP = cdiv(s.N * s.OH * s.OW, 16);
    const bool smallc = s.C <= 4;
    const int T = cdiv(s.C, 16) * s.R * s.S;
    const double kSimds = 1024.0, kLat = 700.0, kClk = 2.4e3;  // cycles, cycles/us
    ConvConfig best{1, 1, 1};
    double best_t = 1e30;
    static const int fks[] = {1, 2, 4}, fps[] = {1, 2, 4};
    // A split pays a device-scope release per workgroup (the partials must be
    // visible across XCDs, whose L2s are not coherent), which measured ~20 ns
    // of serialized time per workgroup on MI355X: it never wins at these
    // sizes, so the model only considers unsplit launches for now.
    static const int splits[] = {1};
    for (int fk : fks) {
        if (fk > 1 && fk > KB) continue;
        for (int fp : fps) {
            if (fp > 1 && fp > MP) continue;
            const long tiles = (long)cdiv(MP, fp) * cdiv(KB, fk);
            for (int sp : splits) {
                if (sp > 1 && T / sp < 2 * kWaves) continue;
                const long wgs = tiles * sp;
                const double steps = std::ceil((double)T / sp / kWaves);
                const double mfma_step = (smallc ? 1.0 : 4.0) * fk * fp * 32.0;
                const double waves_per_simd = std::max(1.0, wgs * kWaves / kSimds);
                const double rounds = std::ceil(waves_per_simd / 8.0);
                const double resident = std::min(8.0, waves_per_simd);
                // latency hidden by the prefetch ring and by other resident waves
                const double per_step = std::max(mfma_step * resident, kLat / 4.0);
                double t = rounds * steps * per_step / kClk;
                t += 1.0;  // launch + epilogue
                if (sp > 1) {
                    const double bytes = 2.0 * sp * tiles * fk * fp * 1024.0;
                    t += bytes / 4.0e6 + 0.8;  // ~4 TB/s L2 round trip + last-arrival pass
                }
                if (t < best_t * 0.98) {
                    best_t = t;
                    best = ConvConfig{fk, fp, sp};
                }
            }
        }
    }
    return best;
}

size_t conv_workspace_bytes(const ConvShape& s, const ConvConfig& c) {
    if (c.split <= 1) return 0;
    const long tiles = (long)cdiv(cdiv(s.N * s.OH * s.OW, 16), c.fp) * cdiv(cdiv(s.K, 16), c.fk);
    return (size_t)c.split * tiles * c.fk * c.fp * 1024;
}

size_t conv_counter_count(const ConvShape& s, const ConvConfig& c) {
    if (c.split <= 1) return 0;
    return (size_t)cdiv(cdiv(s.N * s.OH * s.OW, 16), c.fp) * cdiv(cdiv(s.K, 16), c.fk);
}

hipError_t launch_conv2d(const ConvShape& s, const ConvConfig& c, const float* x, const float* w,
                         const float* bias, const float* res, float* y, float* ws, int* cnt,
                         hipStream_t st) {
    ConvArgs a;
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.res = res;
    a.y = y;
    a.ws = ws;
    a.cnt = cnt;
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
    a.split = (c.split > 1 && ws && cnt) ? c.split : 1;
    const bool pw = s.R == 1 && s.S == 1 && s.ph == 0 && s.pw == 0;
    if (s.C <= 4) return dispatch<true, false>(c.fk, c.fp, a, st);
    if (pw) return dispatch<false, true>(c.fk, c.fp, a, st);
    return dispatch<false, false>(c.fk, c.fp, a, st);
}

}  // namespace neo
