// Blocked convolution on fp32 MFMA (gfx950): launch configuration, cost model
// and launcher.  The kernels are in conv_kernel.h; this file instantiates the
// NCHW16c -> NCHW16c family, conv_xy.hip every other pair of blocks.
#include "conv_kernel.h"

namespace neo {

using namespace conv_detail;

static_assert(kMaxGroup == kMaxGroupConvs, "group size");

extern template hipError_t conv_detail::dispatch_all<true>(const ConvConfig&, int, bool, bool,
                                                           const ConvArgs&, hipStream_t);

int conv_group(const ConvShape& s, const ConvConfig& c) {
    if (conv_small_c(s)) return 1;
    const int CB = cdiv(s.C, 16);
    int g = c.fk * c.fp == 1 ? 4 : (c.fk * c.fp == 2 ? 2 : 1);
    while (CB % g) g /= 2;
    return g;
}

int conv_steps(const ConvShape& s, const ConvConfig& c) {
    if (conv_small_c(s)) return s.R * cdiv(s.S, 4);
    return cdiv(s.C, 16) / conv_group(s, c) * s.R * s.S;
}

bool conv_config_valid(const ConvConfig& c) {
    const bool tile = (c.fk == 1 || c.fk == 2 || c.fk == 4) && (c.fp == 1 || c.fp == 2 || c.fp == 4);
    const bool waves = c.waves == 1 || c.waves == 2 || c.waves == 4 ||
                       (c.waves == 8 && c.fk * c.fp <= 4) || (c.waves == 16 && c.fk * c.fp <= 2);
    return tile && waves && c.split >= 1 && c.split <= 64;
}

// Cost model for the launch configuration of one shape, in microseconds: a
// per-launch floor, plus the longest chain of reduction steps any wave walks
// (each step: its MFMAs, or the measured ~300-cycle bookkeeping-and-load
// chain when a SIMD has a single wave, shared between resident waves), plus
// the extra kernel and partial round trip of a split.
ConvConfig choose_conv_config(const ConvShape& s) {
    const int KB = cdiv(s.K, 16), MP = cdiv(s.N * s.OH * s.OW, 16);
    const double kClk = 2400.0;  // cycles per microsecond
    ConvConfig best{1, 1, 1, 4};
    double best_t = 1e30;
    static const int fks[] = {1, 2, 4}, fps[] = {1, 2, 4}, wvs[] = {1, 2, 4, 8, 16};
    static const int splits[] = {1, 2, 3, 4, 6, 8};
    for (int fk : fks) {
        if (fk > 1 && fk > KB) continue;
        for (int fp : fps) {
            if (fp > 1 && fp > MP) continue;
            const long tiles = (long)cdiv(MP, fp) * cdiv(KB, fk);
            for (int wv : wvs) {
                for (int sp : splits) {
                    const ConvConfig c{fk, fp, sp, wv};
                    if (!conv_config_valid(c)) continue;
                    const int T = conv_steps(s, c), G = conv_group(s, c);
                    if (sp > 1 && T / sp < wv) continue;
                    const long wgs = tiles * sp;
                    const double steps = std::ceil((double)T / sp / wv);
                    const double waves_per_simd = (double)wgs * wv / 1024.0;
                    const double resident = std::max(1.0, std::min(8.0, waves_per_simd));
                    const double rounds = std::max(1.0, std::ceil(waves_per_simd / 8.0));
                    const double mfma = 4.0 * G * fk * fp * 32.0;
                    const double chain = 300.0 + 40.0 * (fk + fp);
                    const double per_step = std::max(mfma * resident, chain);
                    double t = 3.5 + rounds * steps * per_step / kClk;
                    if (sp > 1) t += 2.0 + 2.0 * sp * s.N * KB * s.OH * s.OW * 64.0 / 4.0e6;
                    if (t < best_t * 0.98) {
                        best_t = t;
                        best = c;
                    }
                }
            }
        }
    }
    return best;
}

size_t conv_workspace_bytes(const ConvShape& s, const ConvConfig& c) {
    if (c.split <= 1) return 0;
    return (size_t)c.split * s.N * cdiv(s.K, 16) * s.OH * s.OW * 64;
}

namespace {

constexpr long kKFirstMinWgs = 1024;  // launches this large take channel tiles first

// Kernel arguments of one convolution for launch configuration c with G
// channel groups per reduction step.
ConvArgs make_args(const ConvShape& s, const ConvConfig& c, int G, const float* x, const float* w,
                   bool wmfma, const float* bias, const float* res, float* y, float* ws) {
    ConvArgs a;
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.res = res;
    a.y = y;
    a.ws = ws;
    a.N = s.N;
    a.CB = cdiv(s.C, 16);
    a.H = s.H;
    a.W = s.W;
    a.KB = cdiv(s.K, 16);
    a.R = s.R;
    a.S = s.S;
    a.RS = s.R * s.S;
    a.U = cdiv(s.S, 4);
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
    a.CBG = a.CB / G;
    a.T = conv_small_c(s) ? s.R * cdiv(s.S, 4) : a.CBG * s.R * s.S;
    a.split = (c.split > 1 && ws) ? std::min(c.split, a.T) : 1;
    a.xb = s.xb;
    a.XB = cdiv(s.C, s.xb);
    a.xpb = s.xb * 4;
    const int Q = s.xb >= 16 ? s.xb / 16 : 1;
    a.lq = ilog2(Q);
    a.qm = Q - 1;
    a.dblk = s.H * s.W * a.xpb;
    a.yb = s.yb;
    a.lyb = ilog2(s.yb);
    a.KY = cdiv(s.K, s.yb);
    a.KBk = a.KY * s.yb / 16;
    a.x_bytes = (int)((long)s.N * a.XB * s.H * s.W * a.xpb);
    a.w_bytes = (int)((wmfma ? kernel_filter_floats(s) : (long)a.KB * a.CB * a.RS * 256) * 4);
    a.div_ohw = make_fastdiv((unsigned)(s.OH * s.OW));
    a.div_ow = make_fastdiv((unsigned)s.OW);
    a.div_npx = make_fastdiv((unsigned)cdiv(a.M, 16 * c.fp));
    a.div_nkb = make_fastdiv((unsigned)cdiv(a.KBk, c.fk));
    // Large launches take channel tiles first: the workgroups that read one
    // input tile then run on one XCD and share its L2.  Measured on MI355X
    // (tuned, fused plans): from 1024 workgroups up, ResNet-50 batch 32 runs
    // 2.76 ms against 2.82 ms with pixel tiles first, batch 1 and VGG-16
    // batch 1 unchanged; from 512 up, batch 1 is 1.3 % slower.
    a.kfirst = (long)cdiv(a.M, 16 * c.fp) * cdiv(a.KBk, c.fk) >= kKFirstMinWgs;
    a.gap = s.gap;
    return a;
}

}  // namespace

hipError_t launch_conv2d(const ConvShape& s, const ConvConfig& c, const float* x, const float* w,
                         bool wmfma, const float* bias, const float* res, float* y, float* ws,
                         hipStream_t st) {
    if (c.fp == 0) {  // the streaming pointwise kernel (filter in kernel order)
        if (!wmfma || !conv_stream_config_valid(s, c)) return hipErrorInvalidValue;
        return launch_conv_stream(s, c, x, w, bias, res, y, st);
    }
    if (!conv_config_valid(c) || !conv_blocks_valid(s)) return hipErrorInvalidValue;
    if (s.gap && s.N != 1) return hipErrorInvalidValue;
    const int G = conv_group(s, c);
    // a folded global pool writes its sums in the kernel's epilogue: no split
    const ConvArgs a = make_args(s, c, G, x, w, wmfma, bias, res, y, s.gap ? nullptr : ws);
    const bool small = conv_small_c(s);
    if (s.xb == 16 && s.yb == 16) return dispatch_all<false>(c, G, small, wmfma, a, st);
    return dispatch_all<true>(c, G, small, wmfma, a, st);
}

bool conv_group_eligible(const ConvShape& s) {
    return !conv_small_c(s) && s.xb == 16 && s.yb == 16 && !s.gap;
}

int conv_group_steps_min(const ConvShape* s, int n, const ConvConfig& c) {
    int G = 4, steps = 1 << 30;
    for (int i = 0; i < n; ++i) G = std::min(G, conv_group(s[i], c));
    for (int i = 0; i < n; ++i) steps = std::min(steps, cdiv(s[i].C, 16) / G * s[i].R * s[i].S);
    return steps;
}

bool conv_group_config_valid(const ConvShape* s, int n, const ConvConfig& c) {
    if (n < 1 || n > kMaxGroupConvs || c.split != 1 || !conv_config_valid(c)) return false;
    for (int i = 0; i < n; ++i) {
        if (!conv_group_eligible(s[i])) return false;
        const int KB = cdiv(s[i].K, 16), MP = cdiv(s[i].N * s[i].OH * s[i].OW, 16);
        if ((c.fk > 1 && c.fk > KB) || (c.fp > 1 && c.fp > MP)) return false;
    }
    return conv_group_steps_min(s, n, c) >= c.waves;
}

ConvConfig choose_group_config(const ConvShape* s, int n) {
    // the cost model's choice for the member with the most work, made valid
    // for every member (no split, a tile and wave count all can use)
    int big = 0;
    double most = -1;
    for (int i = 0; i < n; ++i) {
        const double f = (double)s[i].N * s[i].OH * s[i].OW * s[i].K * s[i].C * s[i].R * s[i].S;
        if (f > most) {
            most = f;
            big = i;
        }
    }
    ConvConfig c = choose_conv_config(s[big]);
    c.split = 1;
    for (int fk : {c.fk, 2, 1})
        for (int fp : {c.fp, 2, 1})
            for (int wv : {c.waves, 4, 2, 1}) {
                const ConvConfig t{fk, fp, 1, wv};
                if (conv_group_config_valid(s, n, t)) return t;
            }
    return ConvConfig{1, 1, 1, 1};
}

hipError_t launch_conv_group(const ConvShape* s, int n, const ConvConfig& c, const float* const* x,
                             const float* const* w, const float* const* bias,
                             const float* const* res, float* const* y, const GroupPool* pool,
                             hipStream_t st) {
    if (!conv_group_config_valid(s, n, c)) return hipErrorInvalidValue;
    // (a pool with an int8 copy runs in integer group launches only)
    if (pool && (!pow2_block(pool->s.xb) || !pool->x || !pool->y || pool->q.yq)) return hipErrorInvalidValue;
    int G = 4;
    for (int i = 0; i < n; ++i) G = std::min(G, conv_group(s[i], c));
    ConvGroupArgs ga;
    ga.n = n;
    ga.start[0] = 0;
    // Dispatch order: the members with the most reduction steps per tile
    // first (they finish last), ties in the given order.  Each member takes
    // a whole number of rounds over the XCDs.
    int order[kMaxGroup];
    for (int i = 0; i < n; ++i) order[i] = i;
    auto steps = [&](int i) { return cdiv(s[i].C, 16) / G * s[i].R * s[i].S; };
    std::stable_sort(order, order + n, [&](int p, int q) { return steps(p) > steps(q); });
    for (int j = 0; j < n; ++j) {
        const int i = order[j];
        ga.a[j] = make_args(s[i], c, G, x[i], w[i], true, bias[i], res[i], y[i], nullptr);
        ga.cnt[j] = cdiv(ga.a[j].M, 16 * c.fp) * cdiv(ga.a[j].KBk, c.fk);
        ga.start[j + 1] = ga.start[j] + cdiv(ga.cnt[j], kXcds) * kXcds;
    }
    for (int i = n; i < kMaxGroup; ++i) {
        ga.a[i] = ga.a[n - 1];
        ga.cnt[i] = 0;
        ga.start[i + 1] = ga.start[n];
    }
    PoolPart& pp = ga.pool;
    pp = PoolPart{};
    if (pool) {
        const PoolShape& ps = pool->s;
        pp.x = pool->x;
        pp.y = pool->y;
        pp.s = ps;
        pp.CB = cdiv(ps.C, ps.xb);
        pp.lq = ilog2(ps.xb / 4);
        const long total = ((long)ps.N * pp.CB * ps.OH * ps.OW) << pp.lq;
        if (total >= (1L << 31)) return hipErrorInvalidValue;
        pp.total = (int)total;
        pp.max = pool->max ? 1 : 0;
        pp.k33 = ps.R == 3 && ps.S == 3;
        // one output quad per thread, at most 1024 workgroups (then grid-stride)
        const long per = 64L * c.waves;
        pp.wgs = (int)std::min<long>(1024, std::max<long>(1, (total + per - 1) / per));
    }
    return dispatch_group(c, G, ga, ga.start[n] + pp.wgs, st);
}

}  // namespace neo
