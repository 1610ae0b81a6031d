// Internal declarations of libneo: kernel launchers (no validation; the ABI
// layer and the planner validate first) and the error helpers.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstddef>
#include <cstdint>
#include <functional>
#include <string>
#include <vector>

#include "../../include/neo.h"

namespace neo {

// ---- errors -------------------------------------------------------------------------
void set_error(const std::string& msg);
int fail(int code, const std::string& msg);
int hip_fail(hipError_t e, const char* what);

inline int cdiv(int a, int b) { return (a + b - 1) / b; }
// log2 of a power of two
inline int ilog2(int v) {
    int l = 0;
    while ((1 << l) < v) ++l;
    return l;
}
inline bool pow2_block(int b) { return b == 4 || b == 8 || b == 16 || b == 32 || b == 64; }

// ---- convolution ----------------------------------------------------------------------
struct ConvShape {
    int N, C, H, W;      // input (C real channels)
    int K, R, S;         // filter
    int sh, sw, ph, pw;  // stride, pad
    int OH, OW;
    int y_off, y_tot;    // output channel-block view, in blocks of yb
    int act;
    int xb = 16, yb = 16;  // input layout NCHW[xb]c, output (and residual) NCHW[yb]c
    // 1: global average pooling folded in (N = 1): y receives, instead of the
    // outputs, the channel sums of every 16 pixels, [ceil(OH*OW/16)][ceil(K/16)*16]
    int gap = 0;
};

// Launch configuration: register tile (fk channel blocks x fp pixel groups of
// 16 per wave), the number of workgroups the reduction is split over, and the
// waves per workgroup (which split each workgroup's reduction range again).
struct ConvConfig {
    int fk, fp, split, waves;
};
bool conv_config_valid(const ConvConfig& c);
// Inputs with at most 4 channels (network stems) take the small-channel path:
// a reduction step is (filter row r, group u of 4 filter columns) instead of
// (channel block, kernel entry).
inline bool conv_small_c(const ConvShape& s) { return s.C <= 4; }
// Blocks the kernel reads and writes: output 16, 32 or 64; input 16, 32 or 64
// (on the small-channel path, which reads channels 0..3 only, any of 4..64,
// or 1: NCHW1c, which is NCHW itself).
inline bool conv_blocks_valid(const ConvShape& s) {
    const bool yok = s.yb == 16 || s.yb == 32 || s.yb == 64;
    const bool xok = conv_small_c(s) ? (s.xb == 1 || pow2_block(s.xb))
                                     : (s.xb == 16 || s.xb == 32 || s.xb == 64);
    return xok && yok;
}
// Channel blocks per reduction step for a launch configuration (1 on the
// small-channel path), and the reduction steps of one output tile.
int conv_group(const ConvShape& s, const ConvConfig& c);
int conv_steps(const ConvShape& s, const ConvConfig& c);
ConvConfig choose_conv_config(const ConvShape& s);
// Workspace of a split reduction (partial sums of every split), in bytes.
size_t conv_workspace_bytes(const ConvShape& s, const ConvConfig& c);

// Validation and launch configuration shared by the standalone convolution
// entry points: checks every argument (the calling entry point's name `fn`
// leads each error message), then picks the configuration (cost model,
// results database, NEO_CONV_CONFIG override).  On NEO_OK fills the shape,
// the configuration and the residual pointer; nothing is launched.
int conv_prepare(const char* fn, const float* x, int x_block, int N, int C, int H, int W,
                 const float* w_packed, int K, int R, int S, const float* bias, int stride_h,
                 int stride_w, int pad_h, int pad_w, const neo_epilogue* ep, const float* y,
                 int y_block, int y_blk_offset, int y_blk_total, ConvShape* shape,
                 ConvConfig* config, const float** residual);

// Pointwise convolutions as a stream (conv_stream.hip): a launch
// configuration with fp = 0 names the streaming kernel, whose waves keep fk
// output blocks' filter in registers and walk 16-pixel groups, `waves` waves
// per SIMD of the chip.  1x1, stride 1, no padding, NCHW16c in and out, at
// most 8 input blocks, fk x input blocks <= 16; filter in kernel order.  The
// results are bit-identical to the tile kernel with one wave and no split.
bool conv_stream_eligible(const ConvShape& s);
bool conv_stream_config_valid(const ConvShape& s, const ConvConfig& c);
hipError_t launch_conv_stream(const ConvShape& s, const ConvConfig& c, const float* x, const float* w,
                              const float* bias, const float* res, float* y, hipStream_t st);
// A configuration of either kernel, independent of the shape (results files).
inline bool conv_any_config_valid(const ConvConfig& c) {
    const bool stream = c.fp == 0 && c.split == 1 && (c.fk == 1 || c.fk == 2 || c.fk == 4) &&
                        (c.waves == 1 || c.waves == 2 || c.waves == 4 || c.waves == 8);
    return stream || conv_config_valid(c);
}

// Winograd F(2x2, 3x3) convolution (winograd.hip): 3x3, stride 1, NCHW16c in
// and out, more than 4 input channels.  Launch configuration: fk output
// blocks and fp groups of 16 output tiles (2x2 each) per wave, the channel
// blocks split over `split` workgroups (partials, then the direct kernel's
// split reduction) and `waves` waves per workgroup.  u: the transformed filter
// (winograd.h's order, wino_filter_floats floats).
bool wino_eligible(const ConvShape& s);
bool wino_config_valid(const ConvShape& s, const ConvConfig& c);
ConvConfig choose_wino_config(const ConvShape& s);
size_t wino_filter_floats(const ConvShape& s);
void wino_filter_host(const float* w, int K, int C, float* u);
hipError_t launch_wino_filter(const float* w, int K, int C, float* u, hipStream_t st);
hipError_t launch_wino(const ConvShape& s, const ConvConfig& c, const float* x, const float* u,
                       const float* bias, const float* res, float* y, float* ws, hipStream_t st);
// Local search over the Winograd configurations (results database, "wino"
// entries), and the database's configuration for a shape, if any.
int tune_wino(const ConvShape& s, const float* x, const float* u, const float* bias,
              const float* res, float* y, hipStream_t st, ConvConfig* best, float* us);
bool tuned_wino_config(const ConvShape& s, ConvConfig* out);
// The same for the integer conv (configurations of int8_config_valid), keyed
// also by its output mode `out` (0 float32, 2 int8, 3 both).
struct I8Member;
int tune_int8(const I8Member& m, hipStream_t st, ConvConfig* best, float* us);
bool tuned_int8_config(const ConvShape& s, int out, ConvConfig* cfg);

// Integer (INT8) convolution (conv_int8.hip): int8 NCHW16c activations with
// the convolution's zero padding stored as a halo, a
// packed int8 filter with per-output-channel scales, int32 accumulation on
// v_mfma_i32_16x16x64_i8.  Configuration: fk output blocks x fp pixel groups
// per wave, `waves` waves splitting the reduction (split must be 1).
// launch_conv_int8 writes the dequantized float32 output y (with the epilogue
// of s: act, y_off, y_tot), or with `acc` non-null the raw int32 sums, or
// with `yq` non-null that output requantized by 1 / yscale into an int8
// NCHW16c view with a (qph, qpw) halo (with `y` null: the view of s;
// with `y` too: both outputs, the int8 one a whole [N][KB] tensor).
size_t int8_filter_bytes(int K, int C, int R, int S);
// Bytes of the int8 activations with their zero halo: N * ceil(C/16) *
// (H + 2 ph) * (W + 2 pw) * 16.
size_t int8_act_bytes(int N, int C, int H, int W, int ph, int pw);
bool int8_config_valid(const ConvShape& s, const ConvConfig& c);
ConvConfig choose_int8_config(const ConvShape& s);
// max |x| over n floats (x 16-byte aligned), written to *out as the float's
// bit pattern.
hipError_t launch_absmax(const float* x, long n, unsigned* out, hipStream_t st);
hipError_t launch_quantize_int8(const float* x, int N, int C, int H, int W, int ph, int pw, float scale,
                                int8_t* q, hipStream_t st);
hipError_t launch_pack_filter_int8(const float* w, int K, int C, int R, int S, int8_t* wq, float* wscale,
                                   hipStream_t st);
// x carries a zero halo of (xph, xpw), at least the conv's padding (-1: the
// padding itself), so one int8 copy serves convs of different paddings.
hipError_t launch_conv_int8(const ConvShape& s, const ConvConfig& c, const int8_t* x, const int8_t* w,
                            const float* wscale, float xscale, const float* bias, const float* res,
                            float* y, int* acc, int8_t* yq, float yscale, int qph, int qpw,
                            hipStream_t st, int xph = -1, int xpw = -1);

// Launch the blocked convolution.  x: NCHW[xb]c; w: KCRS[16]c[16]k, or with
// wmfma the kernel's own filter order (to_kernel_order); bias: [ceil(K/16)*16]
// or null; res: NCHW[yb]c [N][ceil(K/yb)][OH][OW][yb] or null; y: NCHW[yb]c
// view (padding lanes of the last block written as 0).  ws: workspace of at
// least conv_workspace_bytes (a split is only used when it is given).  x and w
// must each be below 2 GiB.
hipError_t launch_conv2d(const ConvShape& s, const ConvConfig& c, const float* x, const float* w,
                         bool wmfma, const float* bias, const float* res, float* y, float* ws,
                         hipStream_t st);

// Pooling on NCHW[xb]c (xb in 4..64); y_off / y_tot: output view in blocks.
struct PoolShape {
    int N, C, H, W, R, S, sh, sw, ph, pw, OH, OW, y_off, y_tot;
    int xb = 16;
};

// An int8 copy of a pooling step's output (block 16 only): int8 NCHW16c
// with a (qph, qpw) zero halo, [N][ceil(C/16)][OH + 2 qph][OW + 2 qpw][16],
// each value clamp(round_half_even(y / scale), -127, 127) with the division
// in float32 (the quantization pass's arithmetic); yq null: none.
struct PoolQ {
    int8_t* yq = nullptr;
    float scale = 1.f;
    int qph = 0, qpw = 0;
    int q_off = 0, q_tot = 0;  // the output's blocks [q_off, q_off + CB) of q_tot (0: CB)
};

// A pooling step run by the last workgroups of a fused conv launch (it is
// independent of the launch's convs); q: its int8 copy (integer group
// launches only), y may then be null.
struct GroupPool {
    PoolShape s;
    bool max;
    const float* x;
    float* y;
    PoolQ q{};
};

// Several independent convolutions in one launch (horizontal fusion): NCHW16c
// in and out, more than 4 input channels, one launch configuration for all
// (no split).  x[i], w[i] (kernel filter order), bias[i], res[i], y[i] as for
// launch_conv2d; pool (may be null) runs in extra workgroups of the launch.
constexpr int kMaxGroupConvs = 4;
bool conv_group_eligible(const ConvShape& s);
bool conv_group_config_valid(const ConvShape* s, int n, const ConvConfig& c);
ConvConfig choose_group_config(const ConvShape* s, int n);
hipError_t launch_conv_group(const ConvShape* s, int n, const ConvConfig& c, const float* const* x,
                             const float* const* w, const float* const* bias,
                             const float* const* res, float* const* y, const GroupPool* pool,
                             hipStream_t st);
// Several independent integer convolutions in one launch: each member's
// operands and outputs as for launch_conv_int8 (y and/or yq; no raw sums),
// one configuration valid for every member; pool (may be null, block 16)
// runs in extra workgroups of the launch.
struct I8Member {
    ConvShape s;
    const int8_t* x;
    const int8_t* w;
    const float* wscale;
    float xscale;
    const float* bias;
    const float* res;
    float* y;
    int8_t* yq;
    float yscale;
    int qph, qpw;
    int xph, xpw;  // the halo of x, at least the conv's padding
    // yq's view in blocks: [q_off, q_off + KB) of q_tot (-1: the view of s
    // when y is null, else the whole [N][KB] tensor)
    int q_off, q_tot;
    // requantize by division by yscale (the quantization pass's arithmetic)
    // instead of by its float32 reciprocal
    bool ydivide = false;
};
// Integer dense layer: xq int8 [N][INp] (INp = dense_i8_row_bytes(IN), rows
// zero-padded), wq int8 [OUT][INp] with per-row scales, exact int32 dot
// products, the conv's float32 epilogue (bias, act) into y [N][OUT] and/or
// requantized by 1 / yscale into yq int8 [N][dense_i8_row_bytes(OUT)].
size_t dense_i8_row_bytes(int IN);
hipError_t launch_pack_dense_int8(const float* w, int OUT, int IN, int8_t* wq, float* wscale, hipStream_t st);
hipError_t launch_quantize_rows_int8(const float* x, int N, int IN, float scale, int8_t* q, hipStream_t st);
hipError_t launch_dense_int8(const int8_t* xq, const int8_t* wq, const float* wscale, float xscale,
                             const float* bias, int N, int IN, int OUT, int act, float* y, int8_t* yq,
                             float yscale, hipStream_t st);
// A conv over few input channels as a 1x1 conv: the shape of that 1x1 conv
// (R * S * C channels on the OH x OW map), and the quantization of the conv's
// float32 input x (NCHW16c, or plain NCHW when nchw) into its im2col rows
// (int8 NCHW16c, no halo) by division by scale.
// (the pass stages each 64 output pixels' input rows in LDS: (C R + 1) *
// (63 sw + S) bytes and a 4-byte offset per im2col channel, at most
// kIm2colMaxLds; N and OH at most 65535)
ConvShape im2col_shape(const ConvShape& s);
constexpr size_t kIm2colMaxLds = 32768;
size_t im2col_lds_bytes(const ConvShape& s);
hipError_t launch_im2col_int8(const float* x, bool nchw, const ConvShape& s, float scale, int8_t* q,
                              hipStream_t st);
// One integer conv from a member's operands (float32 and/or int8 outputs).
hipError_t launch_conv_int8_m(const I8Member& m, const ConvConfig& c, hipStream_t st);
bool int8_group_config_valid(const ConvShape* s, int n, const ConvConfig& c);
ConvConfig choose_int8_group_config(const ConvShape* s, int n);
hipError_t launch_conv_int8_group(const I8Member* m, int n, const ConvConfig& c, const GroupPool* pool,
                                  hipStream_t st);
// Local search over the configurations valid for every member of an integer
// group (with its pool, if any), keyed by the members' shapes and output
// modes (0 float32, 2 int8, 3 both) and the pool.
int tune_int8_group(const I8Member* m, int n, const GroupPool* pool, hipStream_t st, ConvConfig* best,
                    float* us);
// Local search over the configurations valid for every member of a group
// (with its pool, if any); results are kept per group of workloads.
int tune_conv_group(const ConvShape* s, int n, const float* const* x, const float* const* w,
                    const float* const* bias, const float* const* res, float* const* y,
                    const GroupPool* pool, hipStream_t st, ConvConfig* best, float* us);
// Time per launch of a pooling step alone (kept in the results database).
int tune_pool(const GroupPool& p, hipStream_t st, float* us);

// A small-channel convolution (a network stem) and the max pooling that
// reads its output, in one launch (conv_pool.hip): the conv's output is kept
// in LDS and only the pooled map is written, NCHW16c with the pool's view
// (p.y_off, p.y_tot).  Configuration: fk channel blocks and fp pixel groups
// per wave, `waves` waves per workgroup, a ty x tx tile of pooled outputs per
// workgroup.  x: NCHW[xb]c (xb = 1: NCHW); w: the kernel order of the small-
// channel path (to_kernel_order); results bit-identical to launch_conv2d with
// one wave and no split followed by launch_maxpool.
struct ConvPoolConfig {
    int fk, fp, waves, ty, tx;
};
bool conv_pool_eligible(const ConvShape& c, const PoolShape& p);
bool conv_pool_config_valid(const ConvShape& c, const PoolShape& p, const ConvPoolConfig& k);
std::vector<ConvPoolConfig> conv_pool_candidates(const ConvShape& c, const PoolShape& p);
ConvPoolConfig choose_conv_pool_config(const ConvShape& c, const PoolShape& p);
hipError_t launch_conv_pool(const ConvShape& c, const PoolShape& p, const ConvPoolConfig& k,
                            const float* x, const float* w, const float* bias, float* y,
                            hipStream_t st);
// Local search over conv_pool_candidates; keeps the fastest with its time.
int tune_conv_pool(const ConvShape& c, const PoolShape& p, const float* x, const float* w,
                   const float* bias, float* y, hipStream_t st, ConvPoolConfig* best, float* us);

// Local search (tune.cpp): the database's configuration for a shape (with its
// blocks), if any; and a search that times every candidate with the given
// buffers on `st` and returns the fastest with its time per launch in us.
bool tuned_config(const ConvShape& s, bool wmfma, ConvConfig* out);
int tune_conv(const ConvShape& s, bool wmfma, const float* x, const float* w, const float* bias,
              const float* res, float* y, hipStream_t st, ConvConfig* best, float* us);

// Two pointwise convolutions in one launch (conv_pair.hip): a (1x1 stride 1,
// NCHW16c, optional residual) whose output y = b's input is also stored, then
// b (1x1 stride 1, no residual).  Shapes with a kernel: 64 -> 256 -> 64 and
// 64 -> 256 -> 128 channels (ceil(C/16) = 4, 16, 4 or 8).  Filters in kernel
// order.
bool conv_pair_eligible(const ConvShape& a, const ConvShape& b);
hipError_t launch_conv_pair(const ConvShape& a, const ConvShape& b, const float* x, const float* wa,
                            const float* ba, const float* res, float* y, const float* wb,
                            const float* bb, float* z, hipStream_t st);
// Time per launch of a pair (results database).
int tune_conv_pair(const ConvShape& a, const ConvShape& b, const float* x, const float* wa,
                   const float* ba, const float* res, float* y, const float* wb, const float* bb,
                   float* z, hipStream_t st, float* us);

// A 3x3 convolution, the pointwise expansion that reads its output and,
// with n = 3, the pointwise reduction after it, in one launch (conv_pair.hip):
// s[0] 3x3 stride 1 pad 1, 64 -> 64 channels (4 blocks each), no residual,
// its output never stored; s[1] 64 -> 256 1x1 with optional residual, its
// output y stored; s[2] as the second conv of a pair, output z.
bool conv_chain_eligible(const ConvShape* s, int n);
hipError_t launch_conv_chain(const ConvShape* s, int n, const float* x, const float* w0, const float* b0,
                             const float* wa, const float* ba, const float* res, float* y,
                             const float* wb, const float* bb, float* z, hipStream_t st);
int tune_conv_chain(const ConvShape* s, int n, const float* x, const float* w0, const float* b0,
                    const float* wa, const float* ba, const float* res, float* y, const float* wb,
                    const float* bb, float* z, hipStream_t st, float* us);

// ---- timing (local search, global search) ----------------------------------------------
// Time per launch of `launch` on `st` (a stream that is not the legacy null
// stream): one warm-up launch (it also surfaces a launch error before
// capture), then `reps` launches captured into a graph, replayed three times
// between two events; the fastest replay counts.
template <typename F>
hipError_t time_launch(F launch, hipStream_t st, hipEvent_t e0, hipEvent_t e1, float* us) {
    const int reps = 10;
    hipError_t e = launch();
    if (e != hipSuccess) return e;
    hipGraph_t g = nullptr;
    hipGraphExec_t ge = nullptr;
    e = hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal);
    for (int i = 0; i < reps && e == hipSuccess; ++i) e = launch();
    hipError_t e2 = hipStreamEndCapture(st, &g);
    if (e == hipSuccess) e = e2;
    if (e == hipSuccess) e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
    if (g) (void)hipGraphDestroy(g);
    float ms = 1e30f;
    for (int r = 0; r < 3 && e == hipSuccess; ++r) {
        e = hipGraphLaunch(ge, st);
        if (e == hipSuccess) e = hipEventRecord(e0, st);
        if (e == hipSuccess) e = hipGraphLaunch(ge, st);
        if (e == hipSuccess) e = hipEventRecord(e1, st);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float t = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
        if (e == hipSuccess) ms = std::min(ms, t);
    }
    if (ge) (void)hipGraphExecDestroy(ge);
    *us = ms * 1000.f / reps;
    return e;
}

struct Events {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    Events() {
        (void)hipEventCreate(&e0);
        (void)hipEventCreate(&e1);
    }
    ~Events() {
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
    }
};

// ---- layout ---------------------------------------------------------------------------
// dst_off / dst_tot: destination channel view in destination units (channels
// for the default layout, blocks for a blocked one), so a transform can write
// into a slice of a concatenation buffer.  Pass 0 and the full extent
// (C, or ceil(C/db)) for a plain destination.
hipError_t launch_layout_transform(const float* src, int sb, float* dst, int db, int N, int C,
                                   int H, int W, int dst_off, int dst_tot, hipStream_t st);
hipError_t launch_pack_filter(const float* w, int K, int C, int R, int S, int ib, int ob,
                              float* out, hipStream_t st);

// ---- pools ----------------------------------------------------------------------------
hipError_t launch_maxpool(const PoolShape& s, const float* x, float* y, hipStream_t st);
hipError_t launch_avgpool(const PoolShape& s, const float* x, float* y, hipStream_t st);
// Pooling on NCHW16c writing the float32 output y (may be null) and/or its
// int8 copy q (the same float32 values quantized).
hipError_t launch_pool_q(const PoolShape& s, bool max, const float* x, float* y, const PoolQ& q,
                         hipStream_t st);
// Max pooling of int8 NCHW16c x8 [N][ceil(C/16)][H][W][16] (no halo) into the
// int8 copy q (q.scale unused): quantization by division is monotone, so the
// max of values quantized with the copy's scale is the quantized max.
hipError_t launch_maxpool_i8(const PoolShape& s, const int8_t* x8, const PoolQ& q, hipStream_t st);
hipError_t launch_gap(const float* x, int xb, int N, int C, int H, int W, float* y, hipStream_t st);
// The global average pool on NCHW16c (C a multiple of 16) writing the means
// y (may be null) and/or their int8 rows yq [N][C], quantized by division.
hipError_t launch_gap_q(const float* x, int N, int C, int H, int W, float* y, int8_t* yq, float scale,
                        hipStream_t st);
// NCHW16c float32 [N][ceil(C/16)][H][W][16] -> the flattened NCHW rows
// (index (c * H + h) * W + w of image n): float32 y [N][C*H*W] (may be
// null) and/or int8 yq [N][dense_i8_row_bytes(C*H*W)], quantized by division.
hipError_t launch_blk_to_rows_int8(const float* x, int N, int C, int H, int W, float* y, int8_t* yq,
                                   float scale, hipStream_t st);

// ---- global layout search (search.cpp) -----------------------------------------------------
struct SearchNode {
    int op = 0;
    std::vector<int> inputs;
    int residual = -1;
    int N = 0, C = 0, H = 0, W = 0;  // shape of the node's value
};
// conv: (node, ic index, oc index) -> time, not finite or < 0 = no candidate;
// transform: (node, from index, to index) -> time.  Indices into kSearchBlocks.
using SearchCost = std::function<double(int, int, int)>;
extern const int kSearchBlocks[NEO_SEARCH_NB];
int search_block_index(int block);
// A transform that leaves the bytes where they are (1x1 map whose channel
// count both blocks divide), unless it writes into a concat slice.
bool layout_alias(int C, int H, int W, int src, int dst, bool into_concat);
// Algorithm 2 over `order` (a topological order of g); ic / oc receive the
// chosen blocks (0 for non-conv nodes), cost the optimum, max_states the
// widest layer of the program.
int layout_search_dp(const std::vector<SearchNode>& g, const std::vector<int>& order,
                     int default_block, const SearchCost& conv_cost, const SearchCost& xform_cost,
                     std::vector<int>* ic, std::vector<int>* oc, double* cost, long* max_states);

// ---- dense ----------------------------------------------------------------------------
hipError_t launch_dense(const float* x, int N, int IN, const float* w, int OUT,
                        const float* bias, int act, float* y, hipStream_t st);
// The same layer on an input that is the mean of `parts` rows of x (row stride
// xstride floats): x_in = scale * (row 0 + row 1 + ...), summed in row order --
// the per-16-pixel sums of a conv with global average pooling folded in.  N = 1,
// IN <= 16384.
hipError_t launch_dense_parts(const float* x, int parts, int xstride, float scale, int IN,
                              const float* w, int OUT, const float* bias, int act, float* y,
                              hipStream_t st);

// ---- host helpers -----------------------------------------------------------------------
void fold_bn_host(const float* w, const float* bias, const float* gamma, const float* beta,
                  const float* mean, const float* var, float eps, int K, int C, int R, int S,
                  float* w_out, float* bias_out);
void pack_filter_host(const float* w, int K, int C, int R, int S, int ib, int ob, float* out);
// Reorder each 16x16 block of a KCRS[16]c[16]k filter from [c][k] to
// [c/4][k][c%4] (in place is not allowed), and back.
void blocks_to_mfma_order(const float* in, long n_blocks, float* out);
void blocks_from_mfma_order(const float* in, long n_blocks, float* out);
// The filter order the kernel reads with wmfma, from and to KCRS[16]c[16]k:
// C > 4: every block in MFMA order (blocks_to_mfma_order);
// C <= 4: [KB][R][ceil(S/4)][4 g][16 k][4 c], filter column s = 4u + g,
//         zero where s >= S.
// kernel_filter_floats is the size of the kernel order in floats.
long kernel_filter_floats(const ConvShape& s);
void to_kernel_order(const float* packed, const ConvShape& s, float* out);
void from_kernel_order(const float* in, const ConvShape& s, float* packed);

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace neo
