// LayoutTransform (Section 3.2) and filter pre-transformation (Section 3.1.1).
//
// Between NCHW and NCHW[x]c, and between NCHW[x]c and NCHW[x']c, for blocks of
// 4..64 channels, one thread moves one 4-channel quad of one pixel: a float4 on
// each blocked side, 4 scalars on the plain side.  The x/4 quads of a pixel
// block are neighbouring lanes, so the blocked side of a wave is 1 KB
// contiguous, the plain side 64-byte runs of channel planes.  Blocks of 1 or 2
// channels use an element-wise path.  All paths are pure permutations plus
// zero fill: bit-exact.
#include "neo_internal.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

// NCHW -> NCHW[X]c, X = 4 << lq; destination view of d_tot blocks from d_off.
__global__ __launch_bounds__(256) void plain_to_blk(const float* __restrict__ src,
                                                    float* __restrict__ dst, int N, int C, int H,
                                                    int W, int CB, int lq, int d_off, int d_tot) {
    const int X = 4 << lq;
    const int total = (N * CB * H * W) << lq;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int q = t & ((1 << lq) - 1);
        const int pix = t >> lq;  // ((n*CB + cb)*H + h)*W + w
        const int w = pix % W;
        int r = pix / W;
        const int h = r % H;
        r /= H;
        const int cb = r % CB;
        const int n = r / CB;
        v4f v;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = cb * X + 4 * q + i;
            v[i] = c < C ? src[((n * C + c) * H + h) * W + w] : 0.f;
        }
        *reinterpret_cast<v4f*>(dst + (((n * d_tot + d_off + cb) * H + h) * W + w) * X + 4 * q) = v;
    }
}

// NCHW[X]c -> NCHW; destination view of c_tot channels from c_off.
__global__ __launch_bounds__(256) void blk_to_plain(const float* __restrict__ src,
                                                    float* __restrict__ dst, int N, int C, int H,
                                                    int W, int CB, int lq, int c_off, int c_tot) {
    const int X = 4 << lq;
    const int total = (N * CB * H * W) << lq;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int q = t & ((1 << lq) - 1);
        const int pix = t >> lq;
        const int w = pix % W;
        int r = pix / W;
        const int h = r % H;
        r /= H;
        const int cb = r % CB;
        const int n = r / CB;
        const v4f v = *reinterpret_cast<const v4f*>(src + pix * X + 4 * q);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = cb * X + 4 * q + i;
            if (c < C) dst[((n * c_tot + c_off + c) * H + h) * W + w] = v[i];
        }
    }
}

// NCHW[XS]c -> NCHW[XD]c (XS = 4 << ls, XD = 4 << ld), one destination quad per
// thread.  A quad never straddles a source block (both are multiples of 4);
// quads at or past C are the destination's zero padding.
__global__ __launch_bounds__(256) void blk_to_blk(const float* __restrict__ src, int ls,
                                                  float* __restrict__ dst, int ld, int N, int C,
                                                  int H, int W, int d_off, int d_tot) {
    const int XS = 4 << ls, XD = 4 << ld;
    const int CBs = (C + XS - 1) / XS, CBd = (C + XD - 1) / XD;
    const int HW = H * W;
    const int total = (N * CBd * HW) << ld;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int q = t & ((1 << ld) - 1);
        const int pix = t >> ld;  // (n*CBd + cbd)*HW + hw
        const int hw = pix % HW;
        const int r = pix / HW;
        const int cbd = r % CBd;
        const int n = r / CBd;
        const int c = cbd * XD + 4 * q;
        v4f v = v4f{0.f, 0.f, 0.f, 0.f};
        if (c < C)
            v = *reinterpret_cast<const v4f*>(src + ((n * CBs + (c >> (ls + 2))) * HW + hw) * XS +
                                              (c & (XS - 1)));
        *reinterpret_cast<v4f*>(dst + ((n * d_tot + d_off + cbd) * HW + hw) * XD + 4 * q) = v;
    }
}

// Element-wise path: one thread per destination element.
__global__ __launch_bounds__(256) void any_to_any(const float* __restrict__ src, int sb,
                                                  float* __restrict__ dst, int db, int N, int C,
                                                  int H, int W, int c_off, int c_tot) {
    const int CBs = sb ? (C + sb - 1) / sb : 0;
    const int Cd = db ? ((C + db - 1) / db) * db : C;
    const int total = N * Cd * H * W;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        int n, c, h, w;
        if (db) {
            const int ci = t % db;
            int r = t / db;
            w = r % W;
            r /= W;
            h = r % H;
            r /= H;
            const int CBd = Cd / db;
            const int cbd = r % CBd;
            n = r / CBd;
            c = cbd * db + ci;
        } else {
            w = t % W;
            int r = t / W;
            h = r % H;
            r /= H;
            c = r % C;
            n = r / C;
        }
        float v = 0.f;
        if (c < C) {
            if (sb)
                v = src[(((n * CBs + c / sb) * H + h) * W + w) * sb + c % sb];
            else
                v = src[((n * C + c) * H + h) * W + w];
        }
        if (db)
            dst[(((n * c_tot + c_off + c / db) * H + h) * W + w) * db + c % db] = v;
        else
            dst[((n * c_tot + c_off + c) * H + h) * W + w] = v;
    }
}

__global__ __launch_bounds__(256) void pack_kernel(const float* __restrict__ w, int K, int C,
                                                   int R, int S, int ib, int ob,
                                                   float* __restrict__ out) {
    const int KB = (K + ob - 1) / ob, CB = (C + ib - 1) / ib;
    const int total = KB * CB * R * S * ib * ob;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int ko = t % ob;
        int r_ = t / ob;
        const int ci = r_ % ib;
        r_ /= ib;
        const int s = r_ % S;
        r_ /= S;
        const int r = r_ % R;
        r_ /= R;
        const int cb = r_ % CB;
        const int kb = r_ / CB;
        const int k = kb * ob + ko, c = cb * ib + ci;
        out[t] = (k < K && c < C) ? w[((k * C + c) * R + r) * S + s] : 0.f;
    }
}

inline dim3 grid_for(long total) {
    long b = (total + 255) / 256;
    if (b > 65536) b = 65536;
    if (b < 1) b = 1;
    return dim3((unsigned)b);
}

}  // namespace

hipError_t launch_layout_transform(const float* src, int sb, float* dst, int db, int N, int C,
                                   int H, int W, int c_off, int c_tot, hipStream_t st) {
    const bool vs = sb == 0 || pow2_block(sb), vd = db == 0 || pow2_block(db);
    if (vs && vd && sb == 0 && db != 0) {
        const int CB = cdiv(C, db), lq = ilog2(db / 4);
        hipLaunchKernelGGL(plain_to_blk, grid_for(((long)N * CB * H * W) << lq), dim3(256), 0, st,
                           src, dst, N, C, H, W, CB, lq, c_off, c_tot);
    } else if (vs && vd && sb != 0 && db == 0) {
        const int CB = cdiv(C, sb), lq = ilog2(sb / 4);
        hipLaunchKernelGGL(blk_to_plain, grid_for(((long)N * CB * H * W) << lq), dim3(256), 0, st,
                           src, dst, N, C, H, W, CB, lq, c_off, c_tot);
    } else if (vs && vd && sb != 0 && db != 0) {
        const int ld = ilog2(db / 4);
        hipLaunchKernelGGL(blk_to_blk, grid_for(((long)N * cdiv(C, db) * H * W) << ld), dim3(256),
                           0, st, src, ilog2(sb / 4), dst, ld, N, C, H, W, c_off, c_tot);
    } else {
        const long Cd = db ? (long)cdiv(C, db) * db : C;
        hipLaunchKernelGGL(any_to_any, grid_for((long)N * Cd * H * W), dim3(256), 0, st, src, sb,
                           dst, db, N, C, H, W, c_off, c_tot);
    }
    return hipGetLastError();
}

hipError_t launch_pack_filter(const float* w, int K, int C, int R, int S, int ib, int ob,
                              float* out, hipStream_t st) {
    const long total = (long)cdiv(K, ob) * ob * cdiv(C, ib) * ib * R * S;
    hipLaunchKernelGGL(pack_kernel, grid_for(total), dim3(256), 0, st, w, K, C, R, S, ib, ob, out);
    return hipGetLastError();
}

}  // namespace neo
