// Internal declarations of libneo: kernel launchers (no validation; the ABI
// layer and the planner validate first) and the error helpers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/neo.h"

namespace neo {

// ---- errors -------------------------------------------------------------------------
void set_error(const std::string& msg);
int fail(int code, const std::string& msg);
int hip_fail(hipError_t e, const char* what);

inline int cdiv(int a, int b) { return (a + b - 1) / b; }

// ---- convolution ----------------------------------------------------------------------
struct ConvShape {
    int N, C, H, W;      // input (C real channels; CB = ceil(C/16) blocks)
    int K, R, S;         // filter
    int sh, sw, ph, pw;  // stride, pad
    int OH, OW;
    int y_off, y_tot;    // output channel-block view
    int act;
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
// Channel blocks per reduction step for a launch configuration (1 on the
// small-channel path), and the reduction steps of one output tile.
int conv_group(const ConvShape& s, const ConvConfig& c);
int conv_steps(const ConvShape& s, const ConvConfig& c);
ConvConfig choose_conv_config(const ConvShape& s);
// Workspace of a split reduction (partial sums of every split), in bytes.
size_t conv_workspace_bytes(const ConvShape& s, const ConvConfig& c);

// Launch the blocked convolution.  x: NCHW16c; w: KCRS[16]c[16]k, or with
// wmfma the kernel's own filter order (to_kernel_order); bias: [KB*16] or null; res: NCHW16c
// [N][KB][OH][OW][16] or null; y: NCHW16c view.  ws: workspace of at least
// conv_workspace_bytes (a split is only used when it is given).  x and w must
// each be below 2 GiB.
hipError_t launch_conv2d(const ConvShape& s, const ConvConfig& c, const float* x, const float* w,
                         bool wmfma, const float* bias, const float* res, float* y, float* ws,
                         hipStream_t st);

// Local search (tune.cpp): the database's configuration for a shape, if any;
// and a search that times every candidate with the given buffers on `st`.
bool tuned_config(const ConvShape& s, bool wmfma, ConvConfig* out);
int tune_conv(const ConvShape& s, bool wmfma, const float* x, const float* w, const float* bias,
              const float* res, float* y, hipStream_t st, ConvConfig* best);

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
struct PoolShape {
    int N, C, H, W, R, S, sh, sw, ph, pw, OH, OW, y_off, y_tot;
};
hipError_t launch_maxpool(const PoolShape& s, const float* x, float* y, hipStream_t st);
hipError_t launch_avgpool(const PoolShape& s, const float* x, float* y, hipStream_t st);
hipError_t launch_gap(const float* x, int N, int C, int H, int W, float* y, hipStream_t st);

// ---- dense ----------------------------------------------------------------------------
hipError_t launch_dense(const float* x, int N, int IN, const float* w, int OUT,
                        const float* bias, int act, float* y, hipStream_t st);

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
