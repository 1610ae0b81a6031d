/*
 * neo.h -- C-ABI of libneo: blocked-layout (NCHW[x]c) CNN inference on
 * MI355X (gfx950).
 *
 * The operations follow the problem statement of "Optimizing CNN Model
 * Inference on CPUs" (NeoCPU):
 *   - the convolution of Section 3.1.1 and its blocked layouts NCHW[x]c for
 *     feature maps and KCRS[x]c[y]k for filters (Algorithm 1's INPUT/OUTPUT);
 *   - the LayoutTransform node of Section 3.2;
 *   - the graph-level plan of Section 3.2, which keeps every convolution in
 *     NCHW[x]c with one constant x and inserts layout transforms only before
 *     the first blocked operation and before layout-dependent operations;
 *   - the global search of Section 3.3.2 (Algorithm 2), which lets every
 *     convolution choose its own input and output blocks (ic_bn, oc_bn) and
 *     pays the layout transforms that choice needs;
 *   - the memory-bound operations the paper fuses into the convolution (bias,
 *     batch norm folded into the weights, residual add, ReLU; Sections 2.2
 *     and 3).
 *
 * Conventions for every call:
 *   - Pointers documented "device" are HIP device pointers owned by the
 *     caller; the library never frees them.  They must be 16-byte aligned.
 *   - Pointers documented "host" are read during the call only.
 *   - Feature maps in NCHW16c are [N][ceil(C/16)][H][W][16] float32 with the
 *     padded channel lanes (c >= C) holding +0.0.  Plain NCHW is
 *     [N][C][H][W].  Filters in KCRS[16]c[16]k are
 *     [ceil(K/16)][ceil(C/16)][R][S][16 (c)][16 (k)], output channel
 *     innermost, zero padded.
 *   - Every device call is asynchronous on `stream` (a hipStream_t; NULL is
 *     the null stream) and never synchronizes.  A kernel fault surfaces at
 *     the caller's next synchronization.
 *   - Return value: NEO_OK (0) or a negative NEO_ERR_* code; on error nothing
 *     was launched and neo_last_error() holds a message.  No exception or
 *     abort crosses the ABI.
 *   - Tensors are limited to 2^31 - 1 elements.
 */
#ifndef NEO_H
#define NEO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum neo_status {
    NEO_OK = 0,
    NEO_ERR_INVALID_ARG = -1, /* null pointer, non-positive size, bad enum */
    NEO_ERR_SHAPE = -2,       /* sizes inconsistent (e.g. empty output)   */
    NEO_ERR_ALIGN = -3,       /* device pointer not 16-byte aligned        */
    NEO_ERR_UNSUPPORTED = -4, /* valid but not implemented (e.g. groups)   */
    NEO_ERR_HIP = -5,         /* HIP runtime error; message has its text   */
    NEO_ERR_OOM = -6,         /* device allocation failed                  */
    NEO_ERR_STATE = -7        /* object destroyed, or wrong kind of plan   */
};

typedef void* neo_stream_t; /* hipStream_t */

enum neo_act { NEO_ACT_NONE = 0, NEO_ACT_RELU = 1 };

/* Channel block of the blocked layout used by every kernel: 16 fp32 lanes =
 * 64 bytes per pixel block, so two neighbouring pixels fill one 128-byte line. */
#define NEO_BLOCK 16

/* Epilogue fused into the convolution (Sections 2.2 and 3: bias, folded batch
 * norm, element-wise add and activation are fused into the CONV):
 *   y = act(conv + bias[k] + residual)
 * `residual`: NULL, or a device NCHW16c tensor with the output's shape
 * [N][ceil(K/16)][OH][OW][16] (contiguous, no channel view). */
typedef struct neo_epilogue {
    int act;               /* enum neo_act */
    const float* residual; /* device, or NULL */
} neo_epilogue;

/*
 * Convolution over NCHW16c (Section 3.1.1, Algorithm 1):
 *   y[n][k][oh][ow] = act( sum_{c<C, r<R, s<S}
 *        x[n][c][oh*stride_h - pad_h + r][ow*stride_w - pad_w + s] * w[k][c][r][s]
 *        + bias[k] + residual[n][k][oh][ow] )
 * with x taken as zero outside the input (cross-correlation, zero padding),
 * OH = (H + 2 pad_h - R) / stride_h + 1 and OW likewise (floor).
 *
 *   x        device NCHW16c [N][ceil(C/16)][H][W][16]
 *   w_packed device KCRS[16]c[16]k, as written by neo_pack_filter(.., 16, 16, ..)
 *   bias     device [ceil(K/16)*16] (zero padded) or NULL
 *   ep       host, may be NULL (= no activation, no residual)
 *   y        device NCHW16c with `y_cblk_total` channel blocks; the K output
 *            channels are written to blocks [y_cblk_offset, y_cblk_offset +
 *            ceil(K/16)), so a producer can write straight into a slice of a
 *            channel concatenation.  Pass 0 and ceil(K/16) for a plain output.
 * Dilation and groups are 1.  Returns NEO_ERR_SHAPE if OH or OW < 1.
 * The padded output lanes (k >= K) are written as +0.0 (ReLU keeps them 0).
 */
int neo_conv2d_blocked(const float* x, int N, int C, int H, int W, const float* w_packed, int K,
                       int R, int S, const float* bias, int stride_h, int stride_w, int pad_h,
                       int pad_w, const neo_epilogue* ep, float* y, int y_cblk_offset,
                       int y_cblk_total, neo_stream_t stream);

/*
 * The same convolution with the input in NCHW[x_block]c and the output in
 * NCHW[y_block]c (Section 3.1.1: the output layout NCHW[y]c may use another
 * split factor than the input's NCHW[x]c; Algorithm 1's x and y):
 *   x        device [N][ceil(C/x_block)][H][W][x_block], padding lanes +0.0
 *   y        device NCHW[y_block]c with `y_blk_total` blocks of y_block
 *            channels; the output occupies blocks [y_blk_offset,
 *            y_blk_offset + ceil(K/y_block)); its padding lanes (k >= K) are
 *            written as +0.0
 *   ep->residual  NULL or device [N][ceil(K/y_block)][OH][OW][y_block]
 *   w_packed, bias as for neo_conv2d_blocked (the filter is always
 *            KCRS[16]c[16]k: its block size is the kernel's MFMA tile, not a
 *            property of the feature maps).
 * x_block: 16, 32 or 64; when C <= 4 also 1 (NCHW1c, which is plain NCHW:
 * x is [N][C][H][W]), 4, 8.  y_block: 16, 32 or 64.
 * Other blocks return NEO_ERR_UNSUPPORTED.  The arithmetic does not depend on
 * the blocks: with the same launch configuration (the default cost model does
 * not look at the blocks) results are bit-identical to neo_conv2d_blocked's.
 */
int neo_conv2d_nchwxc(const float* x, int x_block, int N, int C, int H, int W,
                      const float* w_packed, int K, int R, int S, const float* bias, int stride_h,
                      int stride_w, int pad_h, int pad_w, const neo_epilogue* ep, float* y,
                      int y_block, int y_blk_offset, int y_blk_total, neo_stream_t stream);

/*
 * neo_conv2d_blocked for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc).  Same arguments, launch configuration, kernels and results as
 * neo_conv2d_blocked (bit-identical), but it calls no hipMalloc, hipFree or
 * allocating library routine: when the configuration splits the reduction
 * across workgroups, the partial sums go to a fixed device array of
 * NEO_NOALLOC_SCRATCH_BYTES, one per GPU, held from the library's load until
 * the process ends (its address is looked up once per device, on the first
 * call that needs it).
 *   - A call whose split needs more partial-sum storage than that
 *     (split * N * ceil(K/16) * OH * OW * 64 bytes) returns
 *     NEO_ERR_UNSUPPORTED and launches nothing.
 *   - Every call on one GPU shares that GPU's array, so calls that may run
 *     at the same time on one GPU (different streams, not ordered by events)
 *     race on it; calls on one stream are ordered by the stream.  The array
 *     keeps the last call's partials; nothing in it needs to start at zero.
 */
#define NEO_NOALLOC_SCRATCH_BYTES (16 * 1024 * 1024)
int neo_conv2d_blocked_noalloc(const float* x, int N, int C, int H, int W,
                               const float* w_packed, int K, int R, int S, const float* bias,
                               int stride_h, int stride_w, int pad_h, int pad_w,
                               const neo_epilogue* ep, float* y, int y_cblk_offset,
                               int y_cblk_total, neo_stream_t stream);

/*
 * LayoutTransform node (Section 3.2): NCHW <-> NCHW[x]c, or NCHW[x]c ->
 * NCHW[x']c.  A block of 0 means plain NCHW; a block x > 0 means
 * [N][ceil(C/x)][H][W][x] with zero-filled padding lanes.  Blocks: 0, 1, 2,
 * 4, 8, 16, 32, 64.  A pure permutation: bit-exact.  src and dst are device
 * buffers that must not overlap.
 */
int neo_layout_transform(const float* src, int src_block, float* dst, int dst_block, int N,
                         int C, int H, int W, neo_stream_t stream);

/*
 * Filter pre-transformation KCRS -> KCRS[ic_bn]c[oc_bn]k (Section 3.1.1, done
 * once at plan time as Section 3.2 describes for model parameters):
 *   w_packed[k/oc][c/ic][r][s][c%ic][k%oc] = w[k][c][r][s], zero padded.
 * w_kcrs and w_packed are device buffers; ic_bn, oc_bn in {1,2,4,8,16,32,64}.
 * Bit-exact.  neo_conv2d_blocked consumes ic_bn = oc_bn = 16.
 */
int neo_pack_filter(const float* w_kcrs, int K, int C, int R, int S, int ic_bn, int oc_bn,
                    float* w_packed, neo_stream_t stream);

/*
 * Winograd convolution F(2x2, 3x3) -- the fast algorithm the paper leaves as
 * future work beside its direct convolution (Sections 1 and 5); the nested
 * minimal filtering algorithm of Lavin and Gray (2016).  The same result as
 * neo_conv2d_blocked with R = S = 3 and stride 1, computed per 2x2 output
 * tile as A^T [ sum_c (G g G^T) .* (B^T d B) ] A over the tile's 4x4 input
 * patch d, with
 *   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1],
 *   G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1],
 *   A^T = [1 1 1 0; 0 1 -1 -1]:
 * 4 multiplications per output and input channel instead of 9.  The rounding
 * differs from the direct sum's (results agree within float32 tolerance, not
 * bit for bit).
 *
 * neo_winograd_filter: the transformed filter U = G g G^T of a KCRS
 * [K][C][3][3] filter, computed in double and rounded once, zero padded:
 * ceil(K/16) * ceil(C/16) * 16 * 256 floats, block (kb, cb, e) for element
 * e = 4i + j of the 4x4 tile holding U[k][c] at ((c%16)/4 * 16 + k%16) * 4 +
 * c%4.  w_kcrs and u are device buffers.
 *
 * neo_conv2d_winograd: x, bias, ep, y and the output view as for
 * neo_conv2d_blocked (NCHW16c), u from neo_winograd_filter; pads >= 0 with
 * OH = H + 2 pad_h - 2 >= 1 (and OW).  C must exceed 4 (smaller inputs are
 * network stems: NEO_ERR_UNSUPPORTED).  Like neo_conv2d_blocked it may split
 * the reduction over workgroups, with the same per-stream workspace (grown
 * outside stream capture only).
 */
int neo_winograd_filter(const float* w_kcrs, int K, int C, float* u, neo_stream_t stream);
int neo_conv2d_winograd(const float* x, int N, int C, int H, int W, const float* u, int K,
                        const float* bias, int pad_h, int pad_w, const neo_epilogue* ep, float* y,
                        int y_cblk_offset, int y_cblk_total, neo_stream_t stream);

/*
 * Integer (INT8) convolution -- the paper's other future work (Sections 1 and
 * 5, integer inference), with the usual symmetric linear quantization (the
 * paper gives no scheme):
 *   activations  q_x = clamp(round_half_even(x / x_scale), -127, 127), one
 *                scale per tensor, the division in float32;
 *   filters      w_scale[k] = max |w[k][:][:][:]| / 127 (1 for an all-zero
 *                output channel), q_w = clamp(round_half_even(w / w_scale[k]));
 *   convolution  acc[n][k][oh][ow] = sum_{c,r,s} q_x * q_w, exact in int32
 *                (the same windows, strides and zero padding as
 *                neo_conv2d_blocked; |acc| <= 127^2 * C * R * S must stay below
 *                2^31, i.e. C * R * S <= 133,000);
 *   output       y = act(acc * (x_scale * w_scale[k]) + bias[k] + residual) in
 *                float32 (the product x_scale * w_scale[k] rounded to float32).
 *
 * neo_quantize_int8: x device fp32 NCHW16c [N][ceil(C/16)][H][W][16] -> xq
 *   device int8 NCHW16c with the zero padding of the convolution that reads
 *   it stored as a halo: [N][ceil(C/16)][H + 2 pad_h][W + 2 pad_w][16], the
 *   pixel (h, w) at (h + pad_h, w + pad_w), halo and padding lanes 0;
 *   x_scale > 0.
 * neo_pack_filter_int8: w_kcrs device fp32 [K][C][R][S] -> w_packed device
 *   int8, int8_filter_bytes = ceil(K/16) * ceil(C/64) * R * S * 1024 bytes,
 *   block (kb, r, s, cg) holding for lane (k, g) the 16 bytes
 *   q_w[16 kb + k][64 cg + 16 g + b][r][s], b = 0..15 (zero padded); and
 *   w_scale device [ceil(K/16)*16] (padding channels 1).
 * neo_conv2d_int8: xq, w_packed and w_scale as written above, xq quantized
 *   with this call's pad_h and pad_w (H and W name the unpadded size); bias device
 *   [ceil(K/16)*16] or NULL; ep, y and the output view as for
 *   neo_conv2d_blocked (float32 NCHW16c).
 * neo_conv2d_int8_acc: the same convolution, writing the raw int32 sums to acc
 *   device [N][ceil(K/16)][OH][OW][16] (padding channels 0): the exact part.
 * neo_conv2d_int8_q: the same float32 value requantized for the next layer,
 *   q = clamp(round_half_even(y * r), -127, 127) with r = 1 / y_scale rounded
 *   to float32 and the product in float32, into yq: device int8 NCHW16c with a
 *   halo, blocks [y_cblk_offset, y_cblk_offset + ceil(K/16)) of
 *   [N][y_cblk_total][OH + 2 y_pad_h][OW + 2 y_pad_w][16] (the next conv's
 *   input, y_pad its padding).  The halo is never written: the caller zeroes
 *   yq once.
 * The float32 output is evaluated with one rounding per operation in this
 *   order: float32(acc) * m[k] (m[k] = x_scale * w_scale[k] in float32),
 *   + bias[k], + residual, then the activation (no fused multiply-add).
 * Dilation and groups are 1.  Errors as for neo_conv2d_blocked.
 */
int neo_quantize_int8(const float* x, int N, int C, int H, int W, float x_scale, int pad_h,
                      int pad_w, int8_t* xq, neo_stream_t stream);
int neo_pack_filter_int8(const float* w_kcrs, int K, int C, int R, int S, int8_t* w_packed,
                         float* w_scale, neo_stream_t stream);
int neo_conv2d_int8(const int8_t* xq, int N, int C, int H, int W, const int8_t* w_packed,
                    const float* w_scale, int K, int R, int S, float x_scale, const float* bias,
                    int stride_h, int stride_w, int pad_h, int pad_w, const neo_epilogue* ep,
                    float* y, int y_cblk_offset, int y_cblk_total, neo_stream_t stream);
int neo_conv2d_int8_q(const int8_t* xq, int N, int C, int H, int W, const int8_t* w_packed,
                      const float* w_scale, int K, int R, int S, float x_scale, const float* bias,
                      int stride_h, int stride_w, int pad_h, int pad_w, const neo_epilogue* ep,
                      float y_scale, int y_pad_h, int y_pad_w, int8_t* yq, int y_cblk_offset,
                      int y_cblk_total, neo_stream_t stream);
int neo_conv2d_int8_acc(const int8_t* xq, int N, int C, int H, int W, const int8_t* w_packed, int K,
                        int R, int S, int stride_h, int stride_w, int pad_h, int pad_w, int32_t* acc,
                        neo_stream_t stream);

/*
 * Integer dense (fully connected) layer, the same quantization scheme as the
 * integer conv (integer inference is the paper's future work, Sections 1
 * and 5): y[n][k] = act(float32(acc) * m[k] + bias[k]) with acc[n][k] =
 * sum_i xq[n][i] * w_q[k][i] exact in int32 and m[k] = x_scale * w_scale[k],
 * evaluated one rounding per operation as for neo_conv2d_int8.  Rows are
 * padded with zero bytes to INp = ceil(in_features / 16) * 16.
 * neo_pack_dense_int8: w device fp32 [out_features][in_features] -> w_rows
 *   device int8 [out_features][INp] (clamp(round_half_even(w / w_scale[k]),
 *   -127, 127), the padding 0), w_scale device [out_features] = max |w[k]| /
 *   127 (1 for a zero row).
 * neo_quantize_rows_int8: x device fp32 [N][in_features] -> xq device int8
 *   [N][INp], clamp(round_half_even(x / x_scale), -127, 127) with the
 *   division in float32, the padding bytes written 0; x_scale > 0.
 * neo_dense_int8: xq and w_rows as written above; bias device [out_features]
 *   or NULL; act NEO_ACT_NONE or NEO_ACT_RELU; y device fp32
 *   [N][out_features] and/or (non-NULL) yq device int8
 *   [N][ceil(out_features / 16) * 16]: y requantized for the next dense
 *   layer, clamp(round_half_even(y * r), -127, 127) with r = 1 / y_scale in
 *   float32 (yq's padding bytes are not written: the caller zeroes them
 *   once).  in_features at most 133,144 (the int32 sum's bound).  xq and
 *   w_rows 16-byte aligned (NEO_ERR_ALIGN); NULL or non-positive arguments
 *   NEO_ERR_INVALID_ARG; other errors as for neo_conv2d_blocked.
 */
int neo_pack_dense_int8(const float* w, int out_features, int in_features, int8_t* w_rows, float* w_scale,
                        neo_stream_t stream);
int neo_quantize_rows_int8(const float* x, int N, int in_features, float x_scale, int8_t* xq,
                           neo_stream_t stream);
int neo_dense_int8(const int8_t* xq, int N, int in_features, const int8_t* w_rows, const float* w_scale,
                   int out_features, float x_scale, const float* bias, int act, float* y, float y_scale,
                   int8_t* yq, neo_stream_t stream);

/*
 * Batch-norm folding (inference simplification inherited by the paper,
 * Section 3): with scale[k] = gamma[k] / sqrt(var[k] + eps),
 *   w_out[k][c][r][s] = w[k][c][r][s] * scale[k]
 *   bias_out[k]       = (bias[k] - mean[k]) * scale[k] + beta[k]
 * computed in double and rounded once to float.  All pointers are host;
 * `bias` may be NULL (taken as 0).  w_out may equal w.  Synchronous, CPU only.
 */
int neo_fold_bn(const float* w, const float* bias, const float* gamma, const float* beta,
                const float* mean, const float* var, float eps, int K, int C, int R, int S,
                float* w_out, float* bias_out);

/*
 * Layout-tolerant pooling on NCHW16c (Section 3.2 lists pooling among the
 * operations that handle the blocked layout):
 *   max: y = max over in-bounds taps of the R x S window (padding = -inf)
 *   avg: y = mean over the in-bounds taps (padding excluded from the count)
 * OH = (H + 2 pad_h - R) / stride_h + 1 (floor); pad must be < window.
 * x, y device NCHW16c; y has `y_cblk_total` blocks and receives blocks
 * [y_cblk_offset, y_cblk_offset + ceil(C/16)) (concat slice, as for conv).
 */
int neo_maxpool2d_blocked(const float* x, int N, int C, int H, int W, int R, int S,
                          int stride_h, int stride_w, int pad_h, int pad_w, float* y,
                          int y_cblk_offset, int y_cblk_total, neo_stream_t stream);
int neo_avgpool2d_blocked(const float* x, int N, int C, int H, int W, int R, int S,
                          int stride_h, int stride_w, int pad_h, int pad_w, float* y,
                          int y_cblk_offset, int y_cblk_total, neo_stream_t stream);

/* Global average pool on NCHW16c: y[n][c] = mean over H*W of x[n][c];
 * x device NCHW16c, y device NCHW16c with H = W = 1. */
int neo_global_avgpool_blocked(const float* x, int N, int C, int H, int W, float* y,
                               neo_stream_t stream);

/* The pools on NCHW[block]c for block 4, 8, 16, 32 or 64 (Section 3.2: pooling
 * is layout tolerant, it runs in the layout its input arrives in).  Input and
 * output use the same block; y_blk_offset / y_blk_total count blocks of that
 * size.  Results do not depend on the block. */
int neo_maxpool2d_nchwxc(const float* x, int block, int N, int C, int H, int W, int R, int S,
                         int stride_h, int stride_w, int pad_h, int pad_w, float* y,
                         int y_blk_offset, int y_blk_total, neo_stream_t stream);
int neo_avgpool2d_nchwxc(const float* x, int block, int N, int C, int H, int W, int R, int S,
                         int stride_h, int stride_w, int pad_h, int pad_w, float* y,
                         int y_blk_offset, int y_blk_total, neo_stream_t stream);
int neo_global_avgpool_nchwxc(const float* x, int block, int N, int C, int H, int W, float* y,
                              neo_stream_t stream);

/*
 * Dense (fully connected) layer after Flatten, a layout-dependent operation
 * that consumes the default layout (Section 3.2):
 *   y[n][o] = act( sum_i w[o][i] * x[n][i] + bias[o] )
 * x device [N][IN], w device [OUT][IN] (row-major), bias device [OUT] or
 * NULL, y device [N][OUT].
 */
int neo_dense(const float* x, int N, int IN, const float* w, int OUT, const float* bias,
              int act, float* y, neo_stream_t stream);

/* ------------------------------------------------------------------------------------ */
/* Graph plan (Section 3.2: layout-transformation elimination)                           */
/* ------------------------------------------------------------------------------------ */
enum neo_op {
    NEO_OP_INPUT = 0,   /* the network input, plain NCHW (N, C, H, W of plan_create) */
    NEO_OP_CONV = 1,    /* conv [+ bias] [+ batch norm] [+ residual] [+ act]          */
    NEO_OP_MAXPOOL = 2, /* R x S window, stride, pad                                  */
    NEO_OP_AVGPOOL = 3, /* in-bounds-count average                                    */
    NEO_OP_GAP = 4,     /* global average pool                                        */
    NEO_OP_CONCAT = 5,  /* channel concatenation of inputs[0..n_inputs)               */
    NEO_OP_FLATTEN = 6, /* (N, C, H, W) -> (N, C*H*W), c-major; layout dependent      */
    NEO_OP_DENSE = 7,   /* y = act(W x + b), W [K][in]                                */
    NEO_OP_OUTPUT = 8   /* the network output (one input), returned in plain layout   */
};

/* One operation of a network description.  All pointers are host and are
 * only read during neo_plan_create (the plan keeps its own device copies). */
typedef struct neo_node {
    int op;              /* enum neo_op */
    int n_inputs;
    const int* inputs;   /* ids (indices into the node array) of the inputs */
    int K, R, S;         /* conv: out channels, window; dense: K = out features; pools: R, S */
    int stride_h, stride_w, pad_h, pad_w;
    int act;             /* conv, dense: enum neo_act */
    int residual;        /* conv: id of a node added before the activation, or -1 */
    const float* w;      /* conv: KCRS [K][C][R][S]; dense: [K][in] */
    const float* bias;   /* [K] or NULL */
    const float* bn_gamma, *bn_beta, *bn_mean, *bn_var; /* [K] each, or all NULL */
    float bn_eps;
    /* conv: the scheme's split factors (Section 3.3.1's ic_bn, oc_bn), i.e. the
     * blocks of its input and output layouts; 0 and 0 = the plan's choice (the
     * plan's block, or the global search's).  Both 0 or both set; see
     * neo_conv2d_nchwxc for the blocks allowed.  ic_bn = 1 (C <= 4): the conv
     * reads its input in the default layout NCHW, which NCHW1c is, so no
     * transform is inserted for an NCHW input such as the network's. */
    int ic_bn, oc_bn;
} neo_node;

typedef struct neo_plan neo_plan;

enum neo_plan_flags {
    /* Build the plan on the host only: layouts, transforms, folded and packed
     * parameters and buffer offsets, but no device memory.  Such a plan can be
     * described and its parameters read back, not run. */
    NEO_PLAN_HOST_ONLY = 1,
    /* Transform around every blocked operation instead of keeping the blocked
     * layout between them (the baseline the paper's elimination improves on).
     * Results are bit-identical to the default plan. */
    NEO_PLAN_NAIVE = 2,
    /* neo_run_graph replays a HIP graph of the launch list instead of
     * launching every step from the host.  The graph is captured (on a
     * private stream of the plan) at the first run and again whenever x_nchw
     * or y_out differ from the previous run; a replay is one hipGraphLaunch on
     * the caller's stream.  Results are bit-identical to eager runs. */
    NEO_PLAN_HIPGRAPH = 4,
    /* Local search (Section 3.3.1): at plan creation, time every candidate
     * launch configuration of each convolution workload not yet in the
     * results database on this GPU and keep the fastest (see neo_tune_db_*).
     * Untuned workloads use a cost model.  Needs a device plan. */
    NEO_PLAN_TUNE = 8,
    /* Global search (Section 3.3.2, Algorithm 2): every conv without a given
     * scheme chooses (ic_bn, oc_bn) among its candidates -- the factors of its
     * channel counts that the kernel supports (16, 32, 64; 1 and 4 for an
     * input of at most 4 channels), always including the plan's block -- by the local
     * search's measured time of each scheme plus the measured time of every
     * layout transform the choice implies, minimised over the whole network by
     * neo_layout_search's dynamic program.  Implies NEO_PLAN_TUNE; needs a
     * device plan. */
    NEO_PLAN_GLOBAL_SEARCH = 16,
    /* Horizontal fusion (not in the paper; for batch-1 latency on a GPU,
     * where one small conv cannot fill the device and a launch costs more
     * than its work): the launch list is list-scheduled in rounds -- a step
     * joins the first round after every step that writes storage it reads --
     * and the NCHW16c convs of more than 4 input channels of one round run as
     * one launch (up to 4, in their original order; with sibling convs and
     * parallel branches such as an Inception module's this fuses convs of
     * different inputs), and a pooling step of the round runs in extra
     * workgroups of such a launch (bit-identical to its own kernel).  The
     * members share one launch configuration (tuned for the launch with
     * NEO_PLAN_TUNE, which also takes the pool out, or splits the convs into
     * launches of their own, when that measures faster), so their results
     * match the oracle but are not bit-identical to an ungrouped plan's. */
    NEO_PLAN_GROUP = 32,
    /* Fold a global average pool into its neighbours (not in the paper; one
     * launch less at batch 1): when its input is one image's output of a
     * conv that nothing else reads, and only dense layers read its result
     * (through a flatten), the conv writes the channel sums of every 16 output
     * pixels instead of its outputs, and each dense layer takes their mean as
     * its input.  Results match the oracle but are not bit-identical to an
     * unfolded plan's (the sums run in another order). */
    NEO_PLAN_FUSE_GAP = 64,
    /* Run a pointwise conv and a later pointwise conv that reads its output
     * (1x1, stride 1, NCHW16c; the second without a residual) as one launch
     * where a kernel exists for the pair's channel counts (64 -> 256 -> 64 or
     * 128: a bottleneck's expanding conv and the next one's reducing conv): each
     * workgroup keeps the first conv's output for its 16 pixels in LDS and
     * still stores it.  With NEO_PLAN_TUNE a pair is kept only where it
     * measures faster than its two convs alone.  Not in the paper. */
    NEO_PLAN_FUSE_PAIRS = 128,
    /* Run a 3x3 conv (stride 1, pad 1, 64 -> 64 channels, no residual) whose
     * output only a pointwise conv reads, with that conv and, when the
     * pointwise conv is the first of a pair (NEO_PLAN_FUSE_PAIRS), the pair's
     * second conv, as one launch: a ResNet bottleneck's 3x3, its expanding
     * 1x1 with the residual and the next bottleneck's reducing 1x1 at the
     * 64-channel width.  The 3x3's output stays in LDS and is never stored.
     * With NEO_PLAN_TUNE a chain is kept only where it measures faster than
     * the 3x3 alone plus the best launches of the rest.  Results match the
     * oracle but are not bit-identical to an unchained plan's (the 3x3's sums
     * run in another order).  Not in the paper. */
    NEO_PLAN_FUSE_CHAINS = 256,
    /* A convolution of at most 4 input channels (a network stem) whose
     * output only a max pooling step reads runs with that pooling in one
     * launch: the workgroups stage the input patch and the filter in LDS,
     * keep the conv's output in LDS and write only the pooled map.  The
     * results are those of the conv with one wave per tile followed by the
     * pooling, bit for bit.  With NEO_PLAN_TUNE the fused launch is kept only
     * where it measures faster than the two launches.  Not in the paper: a
     * batch-1 GPU design choice. */
    NEO_PLAN_FUSE_POOL = 512,
    /* Run the 3x3 stride-1 convs that are launched alone (NCHW16c, more than
     * 4 input channels) by Winograd F(2x2, 3x3) (neo_conv2d_winograd: the
     * paper's future work): the plan also prepares each such conv's
     * transformed filter.  With NEO_PLAN_TUNE the local search times the
     * Winograd kernel's configurations beside the direct kernel's and keeps
     * the faster algorithm per conv.  Results match the oracle within the
     * float32 tolerance, not bit for bit. */
    NEO_PLAN_WINOGRAD = 1024,
    /* Integer inference (the paper's future work, Sections 1 and 5): every
     * conv runs as its float32 input quantized with one scale per tensor
     * (neo_quantize_int8, the conv's padding as the halo) followed by the
     * integer convolution with its float32 epilogue (neo_conv2d_int8: bias,
     * residual, activation); filters are the batch-norm-folded ones
     * quantized per output channel on the device at plan creation.  A value
     * that int8 convs read has one int8 copy (shared by those convs, one
     * scale: max|value| / 127), its zero halo the largest padding among
     * them.  When a conv produces the value, that conv's epilogue writes the
     * copy (requantized by the float32 reciprocal of the scale); when a
     * pooling step does, the pool writes it (quantized by division, as the
     * pass would); either beside its float32 output when anything else
     * reads that.  A concatenation whose parts are all conv or pool outputs
     * is assembled by its parts' producers, each writing its slice of the
     * copy with the concatenation's scale.  Otherwise (the network input, a
     * concatenation of concatenations) the first reader runs the
     * quantization pass.  A conv over few input channels (a stem) whose
     * 64-channel reduction steps at least halve that way runs as a 1x1
     * integer conv over its input's im2col rows (channel (r*S + s)*C + c;
     * the same integer sums): its pass writes those rows, from the NCHW
     * network input directly when nothing else reads the input's blocked
     * copy (that layout transform is then not run).  A max pool writing
     * its output's copy from a conv output of at least 16 MiB (float32)
     * that nothing else reads pools in int8: the conv requantizes by
     * division with the pool copy's scale, the pool takes byte maxima (the
     * same bits: that quantization is monotone).  Dense layers run in int8 too: weights quantized
     * per output row, the flattened input one int8 row per image (written by
     * the producing dense layer, requantized, or by the global average pool
     * or the exit of the blocked layout, quantized by division, or by a
     * pass),
     * exact int32 dot products, the same float32 epilogue.  Pools,
     * concatenation and flatten compute in float32 (the average pools and
     * the global average pool sum in double and round the mean once).  The
     * input scales come from neo_plan_calibrate_int8, which must run before
     * the plan does.
     * Convs run in NCHW16c: block 16, and no NAIVE, GLOBAL_SEARCH, WINOGRAD
     * or fusion flag other than NEO_PLAN_GROUP, which puts independent int8
     * convs (and a pooling step) in one launch, as for float32 (one int8
     * configuration for all members; their quantization passes run before
     * the launch, each copy's at its first reader in the grouped order; the
     * results are those of the convs alone, bit for bit).  With
     * NEO_PLAN_TUNE the local search times every int8 configuration of each
     * conv ("int8" lines in the results file) and of each group ("i8group"
     * lines), keeping a group, its convs in one launch with the pool alone,
     * or every conv alone, whichever measures fastest. */
    NEO_PLAN_INT8 = 2048
};

/*
 * Build a plan from `n_nodes` nodes (any order that refers to existing ids;
 * they are sorted topologically) for an input of shape (N, C, H, W):
 * infer each value's layout from the operation categories of Section 3.2
 * (convolution and pooling run in NCHW[block]c, concatenation follows its
 * inputs, flatten/dense/output need the default layout), insert
 * LayoutTransform steps only where a consumer needs another layout, fold
 * batch norm, pre-pack the filters, and allocate device buffers (concat
 * inputs are written in place into channel slices of the concat buffer).
 * `block` (16, 32 or 64) is the split factor of every conv without a scheme
 * of its own (ic_bn = oc_bn = 0) when NEO_PLAN_GLOBAL_SEARCH is not given;
 * layout-tolerant operations run in the layout their input arrives in.  On
 * success *out owns all device memory of the plan.
 */
int neo_plan_create(const neo_node* nodes, int n_nodes, int N, int C, int H, int W, int block,
                    unsigned flags, neo_plan** out);

/* Write a JSON description (values with shape and layout, inserted
 * transforms, steps, buffer bytes) into buf (NUL-terminated, truncated to
 * len).  Returns the full length needed (excluding the NUL), or an error. */
int neo_plan_describe(const neo_plan* plan, char* buf, size_t len);

/* Output shape of the network: dims[0..3] = N, C, H, W (H = W = 1 after a
 * flatten or dense).  Returns NEO_OK. */
int neo_plan_output_shape(const neo_plan* plan, int* dims);

/* Copy a conv node's prepared parameters to host memory: the folded, packed
 * KCRS[16]c[16]k filter (ceil(K/16)*ceil(C/16)*R*S*256 floats) and the folded
 * bias (ceil(K/16)*16 floats).  Either pointer may be NULL.  Synchronous. */
int neo_plan_conv_params(const neo_plan* plan, int node_id, float* w_packed, float* bias);

/*
 * Run the plan: x_nchw device plain NCHW input of the plan's input shape,
 * y_out device plain output of neo_plan_output_shape.  Asynchronous on
 * `stream`; no host synchronization inside.  Not reentrant for one plan
 * (intermediate buffers belong to the plan).
 */
int neo_run_graph(neo_plan* plan, const float* x_nchw, float* y_out, neo_stream_t stream);

/* Run step `step` (0 <= step < number of steps in neo_plan_describe) of the
 * launch list alone, with the same arguments as neo_run_graph; the steps
 * before it must have run for its input to be meaningful.  For timing single
 * layers as the plan launches them. */
int neo_run_step(neo_plan* plan, int step, const float* x_nchw, float* y_out, neo_stream_t stream);

/*
 * Calibrate a NEO_PLAN_INT8 plan on the input x_nchw (device, NCHW; the
 * output goes to y_out as for neo_run_graph): run the plan step by step on
 * `stream` and, just before each conv or dense layer, set its input scale to
 * max|x| / 127 in float32 over its float32 input as this run produced it
 * (1 for an all-zero input; a copy's writer, conv or pool, runs once with
 * its float32 output only for that, then as the plan does; the parts of an
 * assembled concatenation run in float32 only, and again with their slices
 * once the first reader has set the concatenation's scale; the members of a
 * group launch run one by one, which computes the same values).
 * Synchronizes the stream once per int8 layer (the maximum is read back);
 * drops a captured graph, which the next neo_run_graph captures again with
 * the new scales.  neo_plan_describe then lists each int8 layer's "x_scale".  Errors: NEO_ERR_STATE for a plan without
 * NEO_PLAN_INT8 or host-only, NEO_ERR_INVALID_ARG / _ALIGN for the buffers,
 * NEO_ERR_INVALID_ARG for a non-finite activation.
 */
int neo_plan_calibrate_int8(neo_plan* plan, const float* x_nchw, float* y_out, neo_stream_t stream);

/* Free the plan and its device memory (synchronizes the device first).
 * NULL is ignored.  Later use of the handle returns NEO_ERR_STATE. */
void neo_plan_destroy(neo_plan* plan);

/* ------------------------------------------------------------------------------------ */
/* Results database of the local search (Section 3.3.1: results are kept per workload    */
/* and processor type so that a workload is searched once)                               */
/* ------------------------------------------------------------------------------------ */
/* Process-wide table: (GPU architecture, N, C, H, W, K, R, S, strides, pads, filter
 * order, input and output block) -> launch configuration and its measured time;
 * (GPU architecture, the shapes of a fused launch's convs and pooling step) -> the
 * launch's configuration and time; (GPU architecture, a pooling step's shape) -> its
 * time alone; (GPU architecture, the shapes of a pair of pointwise convs, residual) ->
 * the pair's time in one launch; (GPU architecture, the shapes of a 3x3-led chain of two
 * or three convs, residual) -> the chain's time in one launch; (GPU architecture, a stem
 * conv's and its max pooling's shapes) -> the fused launch's configuration and time;
 * (GPU architecture, a 3x3 stride-1 conv's shape) -> its Winograd configuration and time;
 * (GPU architecture, an integer conv's shape and output mode) -> its int8 configuration and
 * time; (GPU architecture, the shapes and output modes of a launch's integer convs and its
 * pooling step) -> the launch's int8 configuration and time.
 * Text file, one entry per line.  save returns the number of entries
 * written, load the number read, size the number held (entries are merged; a malformed
 * line fails the whole load with NEO_ERR_INVALID_ARG). */
int neo_tune_db_save(const char* path);
int neo_tune_db_load(const char* path);
void neo_tune_db_clear(void);
int neo_tune_db_size(void);

/* ------------------------------------------------------------------------------------ */
/* Global search (Section 3.3.2, Algorithm 2), host only                                 */
/* ------------------------------------------------------------------------------------ */
/* Layouts are indexed over the blocks {0 (NCHW), 4, 8, 16, 32, 64}. */
#define NEO_SEARCH_NB 6

/*
 * Choose every conv's scheme (ic_bn, oc_bn) minimising the total of the
 * schemes' execution times and the layout-transform times they imply, for the
 * network `nodes` with input (N, C, H, W), using the plan's layout rules:
 * a conv reads its input in ic_bn and its residual in oc_bn and writes
 * oc_bn; pooling runs in its input's layout (`block` if that is NCHW); a
 * concat takes its first input's layout when every part is a whole number of
 * its blocks (else `block`, else NCHW) and converts the other parts;
 * flatten, dense and the output need NCHW; a value transformed once serves
 * every later reader of that layout; a transform of a 1x1 map whose channel
 * count both blocks divide is free (an alias), except into a concat.
 *   conv_time   host [n_nodes][NB][NB]: conv_time[v][i][j] = time of conv
 *               node v with ic_bn = block i, oc_bn = block j; a negative or
 *               non-finite entry means "not a candidate"; rows of other nodes
 *               are ignored
 *   xform_time  host [n_nodes][NB][NB]: time of transforming node v's value
 *               from block i to block j (non-negative)
 *   ic_bn, oc_bn  host [n_nodes] out: the chosen blocks of each conv (0 for
 *               other nodes).  A conv's ic_bn of 0 means it reads the
 *               default layout; in a plan's nodes that scheme is ic_bn = 1
 *               (and a node's given ic_bn = 1 is block 0 here).
 *   cost        host out (may be NULL): the minimum total
 * The program is Algorithm 2 with, as its memorised state, the layouts of
 * every value still to be read later; it is exact.  It returns
 * NEO_ERR_UNSUPPORTED if the number of states exceeds 2^20 (the paper then
 * switches to an approximate solver), NEO_ERR_SHAPE if no assignment is
 * feasible.  Synchronous, CPU only.
 */
int neo_layout_search(const neo_node* nodes, int n_nodes, int N, int C, int H, int W, int block,
                      const double* conv_time, const double* xform_time, int* ic_bn, int* oc_bn,
                      double* cost);

/* Message of the last failing call on this thread ("" if none). */
const char* neo_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* NEO_H */
