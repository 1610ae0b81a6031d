/*
 * CPU oracle for blocked-layout CNN inference -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously correct definitions of the operations of a CNN
 * forward pass, in the default NCHW layout, accumulating in double precision
 * and rounding once to float32.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this library; the product path never
 * does.  It shares no code with the HIP library.
 *
 * Every function follows the plain definition of the operation; the paper
 * (Section 3.1.1, "Single thread optimization") defines convolution as each
 * kernel sliding over the input feature map along height and width, taking
 * an element-wise product and accumulating, with reduction over input
 * channel, kernel height and kernel width.  It does not flip the kernel
 * (cross-correlation), and it does not state padding; zero padding per axis
 * with a floor output size is used.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

/* Output size of a window of `k` taps with stride `s` over `n` inputs padded
 * by `p` on both sides (floor). */
static int out_size(int n, int k, int s, int p) { return (n + 2 * p - k) / s + 1; }

/*
 * y[n][k][oh][ow] = sum_{c<C, r<R, s<S} x[n][c][oh*sh - ph + r][ow*sw - pw + s] * w[k][c][r][s]
 * with x taken as zero outside [0,H) x [0,W).  Sum in double, one rounding.
 */
void orc_conv2d(const float* x, int N, int C, int H, int W, const float* w, int K, int R,
                int S, int sh, int sw, int ph, int pw, float* y) {
    const int OH = out_size(H, R, sh, ph), OW = out_size(W, S, sw, pw);
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int n = 0; n < N; ++n)
        for (int k = 0; k < K; ++k)
            for (int oh = 0; oh < OH; ++oh)
                for (int ow = 0; ow < OW; ++ow) {
                    double acc = 0.0;
                    for (int c = 0; c < C; ++c)
                        for (int r = 0; r < R; ++r)
                            for (int s = 0; s < S; ++s) {
                                const int ih = oh * sh - ph + r, iw = ow * sw - pw + s;
                                if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                                acc += (double)x[(((size_t)n * C + c) * H + ih) * W + iw] *
                                       (double)w[(((size_t)k * C + c) * R + r) * S + s];
                            }
                    y[(((size_t)n * K + k) * OH + oh) * OW + ow] = (float)acc;
                }
}

/* Max over the window; taps outside the input are ignored (padding = -inf). */
void orc_maxpool2d(const float* x, int N, int C, int H, int W, int R, int S, int sh, int sw,
                   int ph, int pw, float* y) {
    const int OH = out_size(H, R, sh, ph), OW = out_size(W, S, sw, pw);
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c)
            for (int oh = 0; oh < OH; ++oh)
                for (int ow = 0; ow < OW; ++ow) {
                    float m = -INFINITY;
                    for (int r = 0; r < R; ++r)
                        for (int s = 0; s < S; ++s) {
                            const int ih = oh * sh - ph + r, iw = ow * sw - pw + s;
                            if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                            const float v = x[(((size_t)n * C + c) * H + ih) * W + iw];
                            if (v > m) m = v;
                        }
                    y[(((size_t)n * C + c) * OH + oh) * OW + ow] = m;
                }
}

/* Mean over the in-bounds taps of the window (padding excluded from the count). */
void orc_avgpool2d(const float* x, int N, int C, int H, int W, int R, int S, int sh, int sw,
                   int ph, int pw, float* y) {
    const int OH = out_size(H, R, sh, ph), OW = out_size(W, S, sw, pw);
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c)
            for (int oh = 0; oh < OH; ++oh)
                for (int ow = 0; ow < OW; ++ow) {
                    double acc = 0.0;
                    int cnt = 0;
                    for (int r = 0; r < R; ++r)
                        for (int s = 0; s < S; ++s) {
                            const int ih = oh * sh - ph + r, iw = ow * sw - pw + s;
                            if (ih < 0 || ih >= H || iw < 0 || iw >= W) continue;
                            acc += (double)x[(((size_t)n * C + c) * H + ih) * W + iw];
                            ++cnt;
                        }
                    y[(((size_t)n * C + c) * OH + oh) * OW + ow] = (float)(acc / cnt);
                }
}

/* Mean over all H*W positions of each (n, c) plane. */
void orc_global_avgpool(const float* x, int N, int C, int H, int W, float* y) {
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c) {
            double acc = 0.0;
            for (int i = 0; i < H * W; ++i) acc += (double)x[((size_t)n * C + c) * H * W + i];
            y[(size_t)n * C + c] = (float)(acc / (H * W));
        }
}

/* y[n][o] = b[o] + sum_i w[o][i] * x[n][i]; weights stored [out][in]. */
void orc_dense(const float* x, int N, int IN, const float* w, int OUT, const float* b,
               float* y) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int o = 0; o < OUT; ++o) {
            double acc = b ? (double)b[o] : 0.0;
            for (int i = 0; i < IN; ++i)
                acc += (double)w[(size_t)o * IN + i] * (double)x[(size_t)n * IN + i];
            y[(size_t)n * OUT + o] = (float)acc;
        }
}

/* Number of OpenMP threads a parallel region would use (for reporting). */
int orc_num_threads(void) {
    int t = 1;
#pragma omp parallel
    {
#pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            t = omp_get_num_threads();
#endif
        }
    }
    return t;
}

/* Thread count of the following parallel regions (n >= 1), for timing the
 * oracle on a given number of host cores; does not affect any result. */
void orc_set_num_threads(int n) {
#ifdef _OPENMP
    extern void omp_set_num_threads(int);
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
