// LayoutTransform (Section 3.2) and filter pre-transformation (Section 3.1.1).
//
// NCHW <-> NCHW16c has a vectorized path: one thread per (pixel, 4-channel
// quad) moves a float4 on the blocked side and 4 scalars on the plain side,
// so the blocked side is written/read as 1 KB contiguous per wave and the
// plain side as 64-byte runs of one channel plane.  Any other pair of blocks
// (including x -> x') uses an element-wise path.  All paths are pure
// permutations plus zero fill: bit-exact.
#include "neo_internal.h"

namespace neo {
namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void plain_to_b16(const float* __restrict__ src,
                                                    float* __restrict__ dst, int N, int C, int H,
                                                    int W, int CB, int d_off, int d_tot) {
    const int total = N * CB * H * W * 4;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int q = t & 3;
        const int pix = t >> 2;  // ((n*CB + cb)*H + h)*W + w
        const int w = pix % W;
        int r = pix / W;
        const int h = r % H;
        r /= H;
        const int cb = r % CB;
        const int n = r / CB;
        v4f v;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = cb * 16 + 4 * q + i;
            v[i] = c < C ? src[((n * C + c) * H + h) * W + w] : 0.f;
        }
        *reinterpret_cast<v4f*>(dst + (((n * d_tot + d_off + cb) * H + h) * W + w) * 16 + 4 * q) = v;
    }
}

__global__ __launch_bounds__(256) void b16_to_plain(const float* __restrict__ src,
                                                    float* __restrict__ dst, int N, int C, int H,
                                                    int W, int CB, int c_off, int c_tot) {
    const int total = N * CB * H * W * 4;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < total; t += gridDim.x * blockDim.x) {
        const int q = t & 3;
        const int pix = t >> 2;
        const int w = pix % W;
        int r = pix / W;
        const int h = r % H;
        r /= H;
        const int cb = r % CB;
        const int n = r / CB;
        const v4f v = *reinterpret_cast<const v4f*>(src + pix * 16 + 4 * q);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = cb * 16 + 4 * q + i;
            if (c < C) dst[((n * c_tot + c_off + c) * H + h) * W + w] = v[i];
        }
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
    if (sb == 0 && db == 16) {
        const int CB = cdiv(C, 16);
        hipLaunchKernelGGL(plain_to_b16, grid_for((long)N * CB * H * W * 4), dim3(256), 0, st,
                           src, dst, N, C, H, W, CB, c_off, c_tot);
    } else if (sb == 16 && db == 0) {
        const int CB = cdiv(C, 16);
        hipLaunchKernelGGL(b16_to_plain, grid_for((long)N * CB * H * W * 4), dim3(256), 0, st,
                           src, dst, N, C, H, W, CB, c_off, c_tot);
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
