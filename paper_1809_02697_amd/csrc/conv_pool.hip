// A network stem's convolution (at most 4 input channels) and the max
// pooling that reads its output, in one launch, with the input patch and the
// filter staged in LDS.
//
// ResNet-50's stem (3 -> 64 channels, 7x7 / stride 2 at 224x224) and its
// 3x3 / stride 2 max pool are two launches in the plain plan: the conv writes
// a 3.2 MB map that the pool reads back.  Here a workgroup owns a tile of
// pooled outputs (TY x TX pixels, FK channel blocks of 16) of one image:
//   1. it loads the conv outputs' receptive field (the input patch, channels
//      0..3 of each pixel as one float4, zero outside the image) and the
//      filter blocks of its channels into LDS, once;
//   2. its waves compute the conv outputs the pooling windows of the tile
//      cover (the tile's rows and columns plus the windows' overlap, so the
//      rows and columns shared with neighbouring tiles are computed twice),
//      every MFMA operand read from LDS;
//   3. bias and activation are applied in registers and the results kept in
//      LDS, never written to memory;
//   4. each thread takes pooled output quads and writes their maxima.
// The convolution is the small-channel path of the blocked kernel: a
// reduction step is (filter row r, group u of 4 filter columns); lane group g
// supplies column 4u + g, component t (channel t) feeding MFMA k-step t.  The
// steps, their k-steps and the MFMA operands are the blocked kernel's, in the
// same order, so every conv output is bit-identical to that kernel's with one
// wave and no split per tile (operands past the filter's last column are
// multiplied by its zero padding, adding zeros to sums that are never -0).
// The pooling walks the window row by row with the pooling kernel's
// comparison, so the result is bit-identical to pooling that output.
#include "conv_kernel.h"

namespace neo {

using conv_detail::kXcds;
using conv_detail::v4f;
using conv_detail::xcd_order;

namespace {

struct ConvPoolArgs {
    const float* x;
    const float* w;  // kernel order of the small-channel path: block (kb, r, u), 64 float4s
    const float* bias;
    float* y;
    int N, C, H, W, xb, XB;  // input NCHW[xb]c (xb = 1: NCHW)
    int KB, R, U, T, sh, sw, ph, pw, OH, OW, act;
    int PR, PS, psh, psw, pph, ppw, PH, PW, y_off, y_tot;  // max pooling, NCHW16c output view
    int TY, TX, nty, ntx, nkt;
    int prows, pcols;  // patch extent held in LDS (the largest any workgroup needs)
    int slots;         // conv outputs the workgroup can hold (WAVES * FP * 16)
};

// KR, KU: the filter rows and column groups when known at compile time (7 and
// 2 for a 7x7 filter), so the step loop unrolls; 0: from P at run time.
template <int FK, int FP, int WAVES, int KR, int KU>
__global__ __launch_bounds__(WAVES * 64) void conv_pool_small(ConvPoolArgs P) {
    constexpr bool kFixedT = KR > 0;
    const int T = kFixedT ? KR * KU : P.T;
    extern __shared__ v4f lds[];
    v4f* patch = lds;                                 // [prows][pcols] pixels, channels 0..3
    v4f* filt = patch + P.prows * P.pcols;            // [FK][T][64 lanes]
    v4f* tile = filt + FK * P.T * 64;                 // [slots][FK][4 quads]
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, g = lane >> 4;

    // the workgroup's pooled tile: channel tiles fastest, then across, down, image
    int u_ = xcd_order();
    const int kt = u_ % P.nkt;
    u_ /= P.nkt;
    const int tx = u_ % P.ntx;
    u_ /= P.ntx;
    const int ty = u_ % P.nty;
    const int n = u_ / P.nty;
    const int kb0 = kt * FK;
    const int py0 = ty * P.TY, px0 = tx * P.TX;
    const int py1 = min(py0 + P.TY, P.PH), px1 = min(px0 + P.TX, P.PW);
    // conv outputs the tile's windows read: rows [r_lo, r_hi), columns [c_lo, c_hi)
    const int r_lo = max(0, py0 * P.psh - P.pph);
    const int r_hi = min(P.OH, (py1 - 1) * P.psh - P.pph + P.PR);
    const int c_lo = max(0, px0 * P.psw - P.ppw);
    const int c_hi = min(P.OW, (px1 - 1) * P.psw - P.ppw + P.PS);
    const int NC = c_hi - c_lo, NQ = (r_hi - r_lo) * NC;
    // their receptive field: input rows from ih_base, columns from iw_base
    const int ih_base = r_lo * P.sh - P.ph, iw_base = c_lo * P.sw - P.pw;
    const int prows = (r_hi - r_lo - 1) * P.sh + P.R;
    const int pcols = (NC - 1) * P.sw + 4 * P.U;

    // 1. filter blocks and input patch into LDS
    for (int i = tid; i < FK * P.T * 64; i += WAVES * 64) {
        const int f = i / (P.T * 64), rest = i - f * P.T * 64;
        const int kb = kb0 + f;
        filt[i] = kb < P.KB ? *reinterpret_cast<const v4f*>(P.w + ((long)kb * P.T * 64 + rest) * 4)
                            : v4f{0.f, 0.f, 0.f, 0.f};
    }
    for (int i = tid; i < prows * pcols; i += WAVES * 64) {
        const int pr = i / pcols, pc = i - pr * pcols;
        const int ih = ih_base + pr, iw = iw_base + pc;
        v4f v = v4f{0.f, 0.f, 0.f, 0.f};
        if ((unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W) {
            if (P.xb == 1) {
                const float* px = P.x + ((long)n * P.C * P.H + ih) * P.W + iw;
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    if (t < P.C) v[t] = px[(long)t * P.H * P.W];
            } else {
                v = *reinterpret_cast<const v4f*>(P.x + (((long)n * P.XB * P.H + ih) * P.W + iw) * P.xb);
            }
        }
        patch[pr * P.pcols + pc] = v;
    }
    __syncthreads();

    // 2. the wave's conv outputs: pixel groups wave * FP + p of the region
    int bq[FP];
    bool pv[FP];
#pragma unroll
    for (int p = 0; p < FP; ++p) {
        const int q = (wave * FP + p) * 16 + li;
        pv[p] = q < NQ;
        const int qq = pv[p] ? q : 0;
        const int orow = qq / NC, ocol = qq - orow * NC;
        bq[p] = orow * P.sh * P.pcols + ocol * P.sw + g;
    }
    v4f acc[FK][FP];
#pragma unroll
    for (int f = 0; f < FK; ++f)
#pragma unroll
        for (int p = 0; p < FP; ++p) acc[f][p] = v4f{0.f, 0.f, 0.f, 0.f};
    auto step = [&](int st, int off) {
        v4f a[FK], b[FP];
#pragma unroll
        for (int f = 0; f < FK; ++f) a[f] = filt[(f * T + st) * 64 + lane];
#pragma unroll
        for (int p = 0; p < FP; ++p) b[p] = patch[bq[p] + off];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int f = 0; f < FK; ++f)
#pragma unroll
                for (int p = 0; p < FP; ++p)
                    acc[f][p] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[f][t], b[p][t], acc[f][p], 0, 0, 0);
    };
    if (wave * FP * 16 < NQ) {
        if constexpr (kFixedT) {
            // steps (r, u) row by row
#pragma unroll
            for (int st = 0; st < KR * KU; ++st) step(st, (st / KU) * P.pcols + 4 * (st % KU));
        } else {
            int r = 0, u = 0;
            for (int st = 0; st < T; ++st) {
                step(st, r * P.pcols + 4 * u);
                if (++u == P.U) {
                    u = 0;
                    ++r;
                }
            }
        }
    }

    // 3. act(acc + bias) into LDS; lane (li, g) holds channels 4g..4g+3 of pixel li
#pragma unroll
    for (int f = 0; f < FK; ++f) {
        const int kb = kb0 + f;
        const v4f bb = (P.bias && kb < P.KB) ? *reinterpret_cast<const v4f*>(P.bias + kb * 16 + 4 * g)
                                             : v4f{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < FP; ++p) {
            if (!pv[p]) continue;
            v4f o = acc[f][p] + bb;
            if (P.act == NEO_ACT_RELU) {
#pragma unroll
                for (int v = 0; v < 4; ++v) o[v] = o[v] > 0.f ? o[v] : 0.f;
            }
            tile[(((wave * FP + p) * 16 + li) * FK + f) * 4 + g] = o;
        }
    }
    __syncthreads();

    // 4. max pooling of the tile from LDS: one output quad per thread and turn
    const int tw = px1 - px0;
    const int total = (py1 - py0) * tw * FK * 4;
    for (int i = tid; i < total; i += WAVES * 64) {
        const int qd = i & 3;
        const int f = (i >> 2) % FK;
        const int pix = (i >> 2) / FK;
        const int py = py0 + pix / tw, px = px0 + pix % tw;
        const int kb = kb0 + f;
        if (kb >= P.KB) continue;
        const int oh0 = py * P.psh - P.pph, ow0 = px * P.psw - P.ppw;
        v4f m = v4f{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        for (int r = 0; r < P.PR; ++r) {
            const int oh = oh0 + r;
            if ((unsigned)oh >= (unsigned)P.OH) continue;
            for (int c = 0; c < P.PS; ++c) {
                const int ow = ow0 + c;
                if ((unsigned)ow >= (unsigned)P.OW) continue;
                const v4f v = tile[(((oh - r_lo) * NC + (ow - c_lo)) * FK + f) * 4 + qd];
#pragma unroll
                for (int k = 0; k < 4; ++k) m[k] = v[k] > m[k] ? v[k] : m[k];
            }
        }
        *reinterpret_cast<v4f*>(
            P.y + ((((long)n * P.y_tot + P.y_off + kb) * P.PH + py) * P.PW + px) * 16 + 4 * qd) = m;
    }
}

// Extents of the largest region any workgroup of a tile shape covers.
struct Extents {
    int rows, cols, prows, pcols;
};

Extents extents(const ConvShape& c, const PoolShape& p, int ty, int tx) {
    Extents e;
    e.rows = std::min(c.OH, (ty - 1) * p.sh + p.R);
    e.cols = std::min(c.OW, (tx - 1) * p.sw + p.S);
    e.prows = (e.rows - 1) * c.sh + c.R;
    e.pcols = (e.cols - 1) * c.sw + 4 * cdiv(c.S, 4);
    return e;
}

size_t lds_bytes(const ConvShape& c, const ConvPoolConfig& k, const Extents& e) {
    const int T = c.R * cdiv(c.S, 4);
    return ((size_t)e.prows * e.pcols + (size_t)k.fk * T * 64 + (size_t)k.waves * k.fp * 16 * k.fk * 4) * 16;
}

constexpr size_t kMaxLds = 64 * 1024;

template <int FK, int FP, int WAVES>
hipError_t launch_t(const ConvPoolArgs& a, size_t lds, int wgs, hipStream_t st) {
    if (a.R == 7 && a.U == 2)  // a 7x7 filter: the step loop unrolled
        hipLaunchKernelGGL((conv_pool_small<FK, FP, WAVES, 7, 2>), dim3(wgs), dim3(WAVES * 64), lds, st, a);
    else
        hipLaunchKernelGGL((conv_pool_small<FK, FP, WAVES, 0, 0>), dim3(wgs), dim3(WAVES * 64), lds, st, a);
    return hipGetLastError();
}

// The instantiated kernels: (fk, fp, waves).
constexpr int kKernels[][3] = {{1, 1, 8}, {1, 1, 10}, {1, 1, 16}, {1, 2, 4}, {1, 2, 5},
                               {1, 2, 8}, {2, 1, 8},  {2, 1, 10}, {2, 2, 5}};

}  // namespace

bool conv_pool_eligible(const ConvShape& c, const PoolShape& p) {
    return conv_small_c(c) && c.yb == 16 && !c.gap && c.y_off == 0 &&
           (c.xb == 1 || pow2_block(c.xb)) && p.xb == 16 && p.N == c.N && p.C == c.K &&
           p.H == c.OH && p.W == c.OW && p.R >= 1 && p.S >= 1 && p.ph < p.R && p.pw < p.S;
}

bool conv_pool_config_valid(const ConvShape& c, const PoolShape& p, const ConvPoolConfig& k) {
    bool inst = false;
    for (const auto& t : kKernels) inst |= t[0] == k.fk && t[1] == k.fp && t[2] == k.waves;
    if (!inst || k.ty < 1 || k.tx < 1 || !conv_pool_eligible(c, p)) return false;
    if (k.fk > 1 && cdiv(c.K, 16) % k.fk) return false;
    const Extents e = extents(c, p, k.ty, k.tx);
    return e.rows * e.cols <= k.waves * k.fp * 16 && lds_bytes(c, k, e) <= kMaxLds;
}

std::vector<ConvPoolConfig> conv_pool_candidates(const ConvShape& c, const PoolShape& p) {
    std::vector<ConvPoolConfig> out;
    for (const auto& t : kKernels)
        for (int ty : {1, 2, 3, 4, 6, 8})
            for (int tx : {2, 4, 7, 8, 14, 16, 28}) {
                const ConvPoolConfig k{t[0], t[1], t[2], ty, tx};
                if (!conv_pool_config_valid(c, p, k)) continue;
                // keep the tile shapes that fill a kernel's slots best (at least half)
                const Extents e = extents(c, p, ty, tx);
                if (2 * e.rows * e.cols < k.waves * k.fp * 16) continue;
                out.push_back(k);
            }
    return out;
}

ConvPoolConfig choose_conv_pool_config(const ConvShape& c, const PoolShape& p) {
    const ConvPoolConfig pref{1, 2, 5, 4, 8};  // ResNet-50's stem at batch 1
    if (conv_pool_config_valid(c, p, pref)) return pref;
    const std::vector<ConvPoolConfig> all = conv_pool_candidates(c, p);
    if (!all.empty()) return all.front();
    return ConvPoolConfig{1, 1, 16, 1, 1};
}

hipError_t launch_conv_pool(const ConvShape& c, const PoolShape& p, const ConvPoolConfig& k,
                            const float* x, const float* w, const float* bias, float* y,
                            hipStream_t st) {
    if (!conv_pool_config_valid(c, p, k)) return hipErrorInvalidValue;
    ConvPoolArgs a;
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.y = y;
    a.N = c.N;
    a.C = c.C;
    a.H = c.H;
    a.W = c.W;
    a.xb = c.xb;
    a.XB = cdiv(c.C, c.xb);
    a.KB = cdiv(c.K, 16);
    a.R = c.R;
    a.U = cdiv(c.S, 4);
    a.T = c.R * a.U;
    a.sh = c.sh;
    a.sw = c.sw;
    a.ph = c.ph;
    a.pw = c.pw;
    a.OH = c.OH;
    a.OW = c.OW;
    a.act = c.act;
    a.PR = p.R;
    a.PS = p.S;
    a.psh = p.sh;
    a.psw = p.sw;
    a.pph = p.ph;
    a.ppw = p.pw;
    a.PH = p.OH;
    a.PW = p.OW;
    a.y_off = p.y_off;
    a.y_tot = p.y_tot;
    a.TY = k.ty;
    a.TX = k.tx;
    a.nty = cdiv(p.OH, k.ty);
    a.ntx = cdiv(p.OW, k.tx);
    a.nkt = a.KB / k.fk;
    const Extents e = extents(c, p, k.ty, k.tx);
    a.prows = e.prows;
    a.pcols = e.pcols;
    a.slots = k.waves * k.fp * 16;
    const size_t lds = lds_bytes(c, k, e);
    const long wgs = (long)c.N * a.nty * a.ntx * a.nkt;
    if (wgs <= 0 || wgs > (1L << 30)) return hipErrorInvalidValue;
    switch (k.fk * 100 + k.fp * 10 + (k.waves == 10 ? 0 : k.waves == 16 ? 6 : k.waves)) {
        case 118: return launch_t<1, 1, 8>(a, lds, (int)wgs, st);
        case 110: return launch_t<1, 1, 10>(a, lds, (int)wgs, st);
        case 116: return launch_t<1, 1, 16>(a, lds, (int)wgs, st);
        case 124: return launch_t<1, 2, 4>(a, lds, (int)wgs, st);
        case 125: return launch_t<1, 2, 5>(a, lds, (int)wgs, st);
        case 128: return launch_t<1, 2, 8>(a, lds, (int)wgs, st);
        case 218: return launch_t<2, 1, 8>(a, lds, (int)wgs, st);
        case 210: return launch_t<2, 1, 10>(a, lds, (int)wgs, st);
        case 225: return launch_t<2, 2, 5>(a, lds, (int)wgs, st);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace neo
