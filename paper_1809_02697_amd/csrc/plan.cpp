// Graph plan and runtime: layout-transformation elimination (Section 3.2) and
// the global layout search (Section 3.3.2).
//
// The planner walks the network in topological order and infers the layout of
// every value from the operation categories of Section 3.2:
//   - convolution: runs in NCHW[x]c, reading its input in NCHW[ic_bn]c and its
//     residual in NCHW[oc_bn]c and writing NCHW[oc_bn]c, where (ic_bn, oc_bn)
//     is its scheme: given by the caller, chosen by the global search, or
//     (block, block) with one constant block for every convolution;
//   - layout tolerant (max/avg pooling, global average pooling): run in the
//     layout their input arrives in (the plan's block if that is NCHW);
//   - layout oblivious (concatenation): takes the layout of its first input
//     when every input is a whole number of its blocks (else the plan's block,
//     else NCHW) and the other inputs are converted to it;
//   - layout dependent (flatten, dense, the network output): default layout.
// A LayoutTransform step is inserted only where a consumer needs a layout the
// value does not have yet (once per value and layout), so with one block a
// CNN gets one transform at its input and one before flatten.  Parameters are
// prepared once (Section 3.2: model parameters are pre-transformed at compile
// time): batch norm folded, filters packed to KCRS[16]c[16]k.  Concatenation
// costs no step: its producers write straight into channel slices of its
// buffer.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <mutex>
#include <queue>
#include <set>
#include <sstream>
#include <string>
#include <vector>

#include "neo_internal.h"

using namespace neo;

namespace {

enum StepKind { ST_TRANSFORM, ST_CONV, ST_MAXPOOL, ST_AVGPOOL, ST_GAP, ST_DENSE, ST_COPY, ST_CONV_GROUP,
                ST_CONV_PAIR, ST_CONV_CHAIN, ST_CONV_POOL };

struct Val {
    int N = 0, C = 0, H = 0, W = 0;
    int layout = 0;     // 0 = NCHW, x > 0 = NCHW[x]c
    int node = -1;      // node whose result this is (a version of it)
    int alias_of = -1;  // shares the storage of this value (identity transform, flatten)
    int buf = -1;       // root buffer, or kExtIn
    int c_off = 0;      // view offset in the root buffer (blocks if blocked, else channels)
    int c_tot = 0;      // channel extent of the root buffer (same unit as c_off)
    bool view = false;  // written into a slice of a concat buffer
    int consumers = 0;
};

constexpr int kExtIn = -2;

struct Step {
    int kind;
    int node;         // originating node (transforms: the consumer that needed it)
    int in = -1, out = -1, res = -1;
    int out2 = -1;    // ST_CONV_PAIR: the second conv's output (out is the first's);
                      // ST_CONV_CHAIN: the third conv's output, if any (out is the second's)
    ConvShape cs{};
    ConvConfig cc{1, 1, 1, 4};
    bool tuned = false;
    PoolShape ps{};
    long w_off = -1, b_off = -1;
    int src_block = 0, dst_block = 0;
    int dense_in = 0, dense_out = 0, act = 0;
    // ST_DENSE fed by a conv with global average pooling folded in: its input
    // value holds gap_parts rows of channel sums (row stride gap_stride floats)
    int gap_parts = 0, gap_stride = 0;
    float gap_scale = 1.f;
    std::vector<Step> members;  // ST_CONV_GROUP: the convs of one launch (cc is the group's);
                                // ST_CONV_PAIR: the two convs, in order;
                                // ST_CONV_CHAIN: the 3x3 and the one or two pointwise convs
    std::vector<Step> pools;    // ST_CONV_GROUP: a pooling step run by the same launch (0 or 1);
                                // ST_CONV_POOL: the max pooling of members[0]'s output
    ConvPoolConfig cpc{1, 2, 5, 4, 8};  // ST_CONV_POOL
    // ST_CONV with NEO_PLAN_WINOGRAD: the transformed filter (when the shape
    // takes the Winograd kernel), whether the step runs it, its configuration
    long u_off = -1;
    bool wino = false;
    ConvConfig wc{1, 1, 1, 1};
    // ST_CONV with NEO_PLAN_INT8: the folded KCRS filter (float offset), the
    // per-channel scales the device packing writes (float offset), the packed
    // int8 filter (byte offset in the int8 arena), the configuration; the
    // int8 copy of the input it reads (qc), whether this step runs that
    // copy's quantization pass, the copy its own epilogue writes (q_out; -1:
    // none) and whether it also writes its float32 output
    bool i8 = false;
    long kcrs_off = -1, ws8_off = -1, w8_off = -1;
    ConvConfig c8{1, 1, 1, 1};
    int qc = -1, q_out = -1;
    bool quant_here = false, f32_needed = true;
    // the slice of copy q_out this step writes, in blocks ([q_off8, q_off8 +
    // its blocks) of q_tot8), when it is one part of a concatenation's copy
    int q_off8 = -1, q_tot8 = -1;
    // ST_MAXPOOL with NEO_PLAN_INT8: pools copy p8, its conv's int8 output
    int p8 = -1;
    // ST_DENSE with NEO_PLAN_INT8 over many images: run as the 1x1 integer
    // conv cs (its filter packed in the conv's order, configuration c8)
    bool d_conv = false;
    // ST_CONV with NEO_PLAN_INT8 over few input channels (a network stem):
    // run as the 1x1 integer conv over the input's im2col rows (R * S * C
    // channels, the filter in K(RS)C order), which sums the same products
    // with far fewer 64-channel reduction steps
    bool i2c = false;
};

// The shape an integer conv step runs.
static ConvShape int8_conv_shape(const Step& s) { return s.i2c ? im2col_shape(s.cs) : s.cs; }

// NEO_PLAN_INT8: the int8 copy of a value, its halo the largest padding of
// the convs that read it, in the int8 arena, with its scale; written by the
// conv or pooling step producing the value (writer) or by one quantization
// pass (run by the first conv that reads it)
struct I8Copy {
    int val, ph, pw;
    long xq_off;
    float xscale = 1.f;
    int writer = -1;
    // a concatenation's copy assembled by its parts' producers, each writing
    // its slice (their steps carry q_out = this copy)
    bool assembled = false;
    // a dense layer's input: int8 rows [N][dense_i8_row_bytes(C)], no halo
    bool rows = false;
    // the im2col rows of one conv's input (the conv's shape), no halo;
    // quantized by that conv's own pass
    bool im2col = false;
    ConvShape ics{};
    // im2col from the plain NCHW value src, whose blocked copy (val) nothing
    // else reads: the layout transform producing val is dropped
    int src = -1;
    // a max pool's input written in int8 by its conv (no halo) for an int8
    // max pool: requantized by division, with the pool's copy's scale
    // (copy pool_copy); set at calibration
    bool divide = false;
    int pool_copy = -1;
};

struct Xform {
    int from_val, to_val, from_layout, to_layout, consumer_node;
    bool alias;
};

struct NodeInfo {
    neo_node nd;
    std::vector<int> inputs;
    int N = 0, C = 0, H = 0, W = 0;
    int val = -1;         // canonical value of the node
    int ic = 0, oc = 0;   // conv scheme (input / output block), 0 = not chosen yet
};

const char* op_name(int op) {
    static const char* names[] = {"input", "conv", "maxpool", "avgpool", "gap",
                                  "concat", "flatten", "dense", "output"};
    return (op >= 0 && op <= 8) ? names[op] : "?";
}

}  // namespace

struct neo_plan {
    unsigned flags = 0;
    int N = 0, C = 0, H = 0, W = 0, block = 16;
    std::vector<NodeInfo> nodes;  // original order
    std::vector<int> order;       // topological order
    std::vector<Val> vals;
    std::vector<Step> steps;
    std::vector<Xform> xforms;
    std::vector<long> buf_bytes, buf_off;
    int ext_out_buf = -1;  // buffer replaced by the caller's output pointer
    long act_bytes = 0;
    std::vector<float> params;  // host copy of prepared parameters
    float* d_params = nullptr;
    char* d_act = nullptr;
    // NEO_PLAN_INT8: int8 arena (packed filters, quantized inputs), whether
    // the input scales have been calibrated, the calibration's maximum word
    long i8_bytes = 0;
    int8_t* d_i8 = nullptr;
    bool i8_ready = false;
    unsigned* d_absmax = nullptr;
    bool i8_f32_out = false;  // calibration: a writer's first run writes float32 only
    std::vector<I8Copy> i8_copies;
    // split-reduction workspace shared by the conv steps (they run in order)
    size_t ws_bytes = 0;
    float* d_ws = nullptr;
    int out_val = -1;
    int out_dims[4] = {0, 0, 0, 0};
    int input_val = -1;
    // NEO_PLAN_HIPGRAPH: captured launch list for (graph_x, graph_y)
    hipStream_t cap_stream = nullptr;
    hipGraphExec_t graph_exec = nullptr;
    const float* graph_x = nullptr;
    float* graph_y = nullptr;
    // NEO_PLAN_GLOBAL_SEARCH: predicted totals (us) of the chosen schemes and of
    // every conv at the plan's block, schemes measured, largest DP layer
    bool searched = false;
    double search_cost = 0, fixed_cost = 0;
    int search_schemes = 0;
    long search_states = 0;
};

static int tune_plan(neo_plan* P);

namespace {

std::mutex g_plans_mu;
std::set<const neo_plan*> g_plans;

bool live(const neo_plan* p) {
    std::lock_guard<std::mutex> lk(g_plans_mu);
    return p && g_plans.count(p);
}

long align_up(long v, long a) { return (v + a - 1) / a * a; }

long val_elems_root(const Val& v) {
    // element count of a full (non-view) buffer holding v
    return v.layout ? (long)v.N * cdiv(v.C, v.layout) * v.layout * v.H * v.W
                    : (long)v.N * v.C * v.H * v.W;
}

int out_dim(int n, int k, int s, int p) { return (n + 2 * p - k) / s + 1; }

// Channel extent of a value in units of its layout (blocks, or channels).
int units(int C, int layout) { return layout ? cdiv(C, layout) : C; }
// A conv's input block 1 (NCHW1c) is the default layout in memory: the conv
// reads that version of its input, and a search choosing the default layout
// for a conv input names it block 1.
int read_layout(int ic) { return ic == 1 ? 0 : ic; }
int scheme_block(int ic) { return ic == 0 ? 1 : ic; }

struct Builder {
    neo_plan* P;
    std::vector<std::map<int, int>> versions;  // node -> layout -> value

    int new_val(int node, int N, int C, int H, int W, int layout) {
        Val v;
        v.N = N; v.C = C; v.H = H; v.W = W;
        v.layout = layout;
        v.node = node;
        P->vals.push_back(v);
        return (int)P->vals.size() - 1;
    }

    // The version of node `nid`'s value in `layout`, inserting a transform
    // (from the node's canonical value) for consumer `consumer` if needed.
    int get(int nid, int layout, int consumer) {
        auto& m = versions[nid];
        auto it = m.find(layout);
        if (it != m.end()) return it->second;
        const int src = P->nodes[nid].val;
        const Val s = P->vals[src];
        const int v = new_val(nid, s.N, s.C, s.H, s.W, layout);
        const bool identity = layout_alias(s.C, s.H, s.W, s.layout, layout,
                                           P->nodes[consumer].nd.op == NEO_OP_CONCAT);
        Xform x{src, v, s.layout, layout, consumer, identity};
        P->xforms.push_back(x);
        if (identity) {
            P->vals[v].alias_of = src;
        } else {
            Step st{};
            st.kind = ST_TRANSFORM;
            st.node = consumer;
            st.in = src;
            st.out = v;
            st.src_block = s.layout;
            st.dst_block = layout;
            P->steps.push_back(st);
        }
        m[layout] = v;
        return v;
    }

    // Register a node's produced value; in a naive plan a blocked result is
    // transformed back to the default layout right away.
    void produce(int nid, int v) {
        const int lay = P->vals[v].layout;
        versions[nid][lay] = v;
        P->nodes[nid].val = v;
        if ((P->flags & NEO_PLAN_NAIVE) && lay != 0) {
            // the blocked result is only read by its transform back; every
            // blocked consumer transforms the default-layout copy again
            const int pv = get(nid, 0, nid);
            P->nodes[nid].val = pv;
            versions[nid].erase(lay);
        }
    }
};

int add_params(neo_plan* P, const std::vector<float>& a) {
    const long off = align_up((long)P->params.size(), 64);
    P->params.resize(off + a.size(), 0.f);
    std::copy(a.begin(), a.end(), P->params.begin() + off);
    return (int)off;
}

// ---- pass 1: validate, copy, order, shapes ----------------------------------------------
// need_params: convs and dense layers must carry weights (a plan); the layout
// search alone needs only the structure.
int parse(neo_plan* P, const neo_node* nodes, int n, bool need_params) {
    int n_in = 0, n_out = 0;
    P->nodes.resize(n);
    for (int i = 0; i < n; ++i) {
        const neo_node& d = nodes[i];
        NodeInfo& ni = P->nodes[i];
        ni.nd = d;
        if (d.op < NEO_OP_INPUT || d.op > NEO_OP_OUTPUT)
            return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": unknown op");
        if (d.n_inputs < 0 || (d.n_inputs > 0 && !d.inputs))
            return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": bad inputs");
        for (int j = 0; j < d.n_inputs; ++j) {
            if (d.inputs[j] < 0 || d.inputs[j] >= n || d.inputs[j] == i)
                return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": input id out of range");
            ni.inputs.push_back(d.inputs[j]);
        }
        const int want = d.op == NEO_OP_INPUT ? 0 : (d.op == NEO_OP_CONCAT ? -1 : 1);
        if ((want >= 0 && d.n_inputs != want) || (want < 0 && d.n_inputs < 1))
            return fail(NEO_ERR_INVALID_ARG, std::string("node ") + std::to_string(i) + " (" +
                                                 op_name(d.op) + "): wrong number of inputs");
        if (d.op == NEO_OP_CONV) {
            if (d.residual < -1 || d.residual >= n || d.residual == i)
                return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": bad residual id");
            if (need_params && !d.w)
                return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": conv without weights");
            const bool any = d.bn_gamma || d.bn_beta || d.bn_mean || d.bn_var;
            const bool all = d.bn_gamma && d.bn_beta && d.bn_mean && d.bn_var;
            if (any && !all)
                return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": partial batch-norm parameters");
            if ((d.ic_bn == 0) != (d.oc_bn == 0))
                return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": ic_bn and oc_bn must both be 0 or both set");
            ni.ic = d.ic_bn;
            ni.oc = d.oc_bn;
        }
        if (need_params && d.op == NEO_OP_DENSE && !d.w)
            return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": dense without weights");
        if ((d.op == NEO_OP_CONV || d.op == NEO_OP_DENSE) && d.act != NEO_ACT_NONE && d.act != NEO_ACT_RELU)
            return fail(NEO_ERR_INVALID_ARG, "node " + std::to_string(i) + ": unknown activation");
        n_in += d.op == NEO_OP_INPUT;
        n_out += d.op == NEO_OP_OUTPUT;
    }
    if (n_in != 1 || n_out != 1)
        return fail(NEO_ERR_INVALID_ARG, "plan needs exactly one input and one output node");

    // topological order (Kahn; ties by node id)
    std::vector<std::vector<int>> succ(n);
    std::vector<int> indeg(n, 0);
    for (int i = 0; i < n; ++i) {
        std::vector<int> deps = P->nodes[i].inputs;
        if (P->nodes[i].nd.op == NEO_OP_CONV && P->nodes[i].nd.residual >= 0)
            deps.push_back(P->nodes[i].nd.residual);
        for (int d : deps) {
            succ[d].push_back(i);
            ++indeg[i];
        }
    }
    std::priority_queue<int, std::vector<int>, std::greater<int>> ready;
    for (int i = 0; i < n; ++i)
        if (!indeg[i]) ready.push(i);
    while (!ready.empty()) {
        const int i = ready.top();
        ready.pop();
        P->order.push_back(i);
        for (int s : succ[i])
            if (--indeg[s] == 0) ready.push(s);
    }
    if ((int)P->order.size() != n) return fail(NEO_ERR_INVALID_ARG, "network has a cycle");

    // shapes
    for (int id : P->order) {
        NodeInfo& ni = P->nodes[id];
        const neo_node& d = ni.nd;
        const std::string where = std::string("node ") + std::to_string(id) + " (" + op_name(d.op) + "): ";
        const NodeInfo* a = ni.inputs.empty() ? nullptr : &P->nodes[ni.inputs[0]];
        switch (d.op) {
            case NEO_OP_INPUT:
                ni.N = P->N; ni.C = P->C; ni.H = P->H; ni.W = P->W;
                break;
            case NEO_OP_CONV:
            case NEO_OP_MAXPOOL:
            case NEO_OP_AVGPOOL: {
                const bool conv = d.op == NEO_OP_CONV;
                if ((conv && d.K <= 0) || d.R <= 0 || d.S <= 0 || d.stride_h <= 0 || d.stride_w <= 0 ||
                    d.pad_h < 0 || d.pad_w < 0)
                    return fail(NEO_ERR_INVALID_ARG, where + (conv ? "bad conv parameters" : "bad pool parameters"));
                if (!conv && (d.pad_h >= d.R || d.pad_w >= d.S))
                    return fail(NEO_ERR_INVALID_ARG, where + "bad pool parameters");
                const int OH = out_dim(a->H, d.R, d.stride_h, d.pad_h);
                const int OW = out_dim(a->W, d.S, d.stride_w, d.pad_w);
                if (a->H + 2 * d.pad_h < d.R || a->W + 2 * d.pad_w < d.S || OH < 1 || OW < 1)
                    return fail(NEO_ERR_SHAPE, where + "empty output");
                ni.N = a->N; ni.C = conv ? d.K : a->C; ni.H = OH; ni.W = OW;
                if (conv && d.residual >= 0) {
                    const NodeInfo* r = &P->nodes[d.residual];
                    if (r->N != ni.N || r->C != ni.C || r->H != ni.H || r->W != ni.W)
                        return fail(NEO_ERR_SHAPE, where + "residual shape differs from the output");
                }
                if (conv && ni.ic) {
                    ConvShape cs{};
                    cs.C = a->C;
                    cs.xb = ni.ic;
                    cs.yb = ni.oc;
                    if (!conv_blocks_valid(cs))
                        return fail(NEO_ERR_UNSUPPORTED, where + "ic_bn / oc_bn not supported by the kernel");
                }
                break;
            }
            case NEO_OP_GAP:
                ni.N = a->N; ni.C = a->C; ni.H = 1; ni.W = 1;
                break;
            case NEO_OP_CONCAT: {
                int C = 0;
                for (int j : ni.inputs) {
                    const NodeInfo* b = &P->nodes[j];
                    if (b->N != a->N || b->H != a->H || b->W != a->W)
                        return fail(NEO_ERR_SHAPE, where + "inputs differ in N, H or W");
                    C += b->C;
                }
                ni.N = a->N; ni.C = C; ni.H = a->H; ni.W = a->W;
                break;
            }
            case NEO_OP_FLATTEN:
                ni.N = a->N; ni.C = a->C * a->H * a->W; ni.H = 1; ni.W = 1;
                break;
            case NEO_OP_DENSE:
                if (a->H != 1 || a->W != 1)
                    return fail(NEO_ERR_SHAPE, where + "input must be flat (insert a flatten)");
                if (d.K <= 0) return fail(NEO_ERR_INVALID_ARG, where + "K must be > 0");
                ni.N = a->N; ni.C = d.K; ni.H = 1; ni.W = 1;
                break;
            case NEO_OP_OUTPUT:
                ni.N = a->N; ni.C = a->C; ni.H = a->H; ni.W = a->W;
                break;
        }
    }
    return NEO_OK;
}

// The network as the layout search sees it.
std::vector<SearchNode> search_nodes(const neo_plan* P) {
    std::vector<SearchNode> g(P->nodes.size());
    for (size_t i = 0; i < P->nodes.size(); ++i) {
        const NodeInfo& ni = P->nodes[i];
        g[i].op = ni.nd.op;
        g[i].inputs = ni.inputs;
        g[i].residual = ni.nd.op == NEO_OP_CONV ? ni.nd.residual : -1;
        g[i].N = ni.N; g[i].C = ni.C; g[i].H = ni.H; g[i].W = ni.W;
    }
    return g;
}

// ---- pass 2: steps, values, buffers --------------------------------------------------------
int build_steps(neo_plan* P) {
    const int n = (int)P->nodes.size();
    Builder B{P, std::vector<std::map<int, int>>(n)};
    const bool naive = P->flags & NEO_PLAN_NAIVE;
    const int D = P->block;
    for (int id : P->order) {
        NodeInfo& ni = P->nodes[id];
        const neo_node& d = ni.nd;
        const std::string where = std::string("node ") + std::to_string(id) + " (" + op_name(d.op) + "): ";
        const NodeInfo* a = ni.inputs.empty() ? nullptr : &P->nodes[ni.inputs[0]];
        // layout of an input as it arrives (its canonical value)
        auto arriving = [&](int j) { return P->vals[P->nodes[ni.inputs[j]].val].layout; };
        switch (d.op) {
            case NEO_OP_INPUT: {
                const int v = B.new_val(id, ni.N, ni.C, ni.H, ni.W, 0);
                P->vals[v].buf = kExtIn;
                P->input_val = v;
                B.versions[id][0] = v;
                ni.val = v;
                break;
            }
            case NEO_OP_CONV: {
                if (!ni.ic) {
                    ni.ic = D;
                    ni.oc = D;
                }
                Step st{};
                st.kind = ST_CONV;
                st.node = id;
                st.in = B.get(ni.inputs[0], read_layout(ni.ic), id);
                if (d.residual >= 0) st.res = B.get(d.residual, ni.oc, id);
                const int C = a->C;
                std::vector<float> w((long)d.K * C * d.R * d.S), b(cdiv(d.K, 16) * 16, 0.f);
                bool has_b = false;
                if (d.bn_gamma) {
                    for (int k = 0; k < d.K; ++k)
                        if (!((double)d.bn_var[k] + (double)d.bn_eps > 0.0))
                            return fail(NEO_ERR_INVALID_ARG, where + "var + eps must be > 0");
                    fold_bn_host(d.w, d.bias, d.bn_gamma, d.bn_beta, d.bn_mean, d.bn_var, d.bn_eps,
                                 d.K, C, d.R, d.S, w.data(), b.data());
                    has_b = true;
                } else {
                    std::copy(d.w, d.w + w.size(), w.begin());
                    if (d.bias) {
                        std::copy(d.bias, d.bias + d.K, b.begin());
                        has_b = true;
                    }
                }
                const long nblk = (long)cdiv(d.K, 16) * cdiv(C, 16) * d.R * d.S;
                if (nblk * 256 >= (1L << 29) ||
                    (long)ni.N * cdiv(C, ni.ic) * ni.ic * a->H * a->W >= (1L << 29))
                    return fail(NEO_ERR_UNSUPPORTED, where + "input or filter of 2 GiB or more");
                st.cs = ConvShape{ni.N, C, a->H, a->W, d.K, d.R, d.S, d.stride_h, d.stride_w,
                                  d.pad_h, d.pad_w, ni.H, ni.W, 0, cdiv(d.K, ni.oc), d.act};
                st.cs.xb = ni.ic;
                st.cs.yb = ni.oc;
                std::vector<float> wp(nblk * 256), wm(kernel_filter_floats(st.cs));
                pack_filter_host(w.data(), d.K, C, d.R, d.S, 16, 16, wp.data());
                to_kernel_order(wp.data(), st.cs, wm.data());  // one float4 per lane and k-quad
                st.w_off = add_params(P, wm);
                if ((P->flags & NEO_PLAN_WINOGRAD) && wino_eligible(st.cs)) {
                    std::vector<float> u(wino_filter_floats(st.cs));
                    if ((long)u.size() >= (1L << 29))
                        return fail(NEO_ERR_UNSUPPORTED, where + "Winograd filter of 2 GiB or more");
                    wino_filter_host(w.data(), d.K, C, u.data());
                    st.u_off = add_params(P, u);
                }
                if (has_b) st.b_off = add_params(P, b);
                if (P->flags & NEO_PLAN_INT8) {
                    if ((long)C * d.R * d.S > 133000)
                        return fail(NEO_ERR_UNSUPPORTED, where + "C * R * S above 133,000 could overflow "
                                                                 "the int32 accumulator");
                    const long xq = (long)int8_act_bytes(ni.N, C, a->H, a->W, d.pad_h, d.pad_w);
                    if ((long)int8_filter_bytes(d.K, C, d.R, d.S) >= (1L << 31) ||
                        xq + 4L * (a->H + 2 * d.pad_h) * (a->W + 2 * d.pad_w) * 16 >= (1L << 31))
                        return fail(NEO_ERR_UNSUPPORTED, where + "int8 input or filter of 2 GiB or more");
                    st.i8 = true;
                    // im2col when it at least halves the reduction steps
                    // (C = 3: 3 instead of 49 for 7x7, 1 instead of 9 for 3x3;
                    // a conv's input is never a concatenation's slice)
                    const long rsc = (long)C * d.R * d.S;
                    st.i2c = d.R * d.S > 1 && P->vals[st.in].layout == 16 && P->vals[st.in].alias_of < 0 &&
                             2 * cdiv(rsc, 64) <= (long)d.R * d.S * cdiv(C, 64) &&
                             (long)int8_act_bytes(ni.N, (int)rsc, ni.H, ni.W, 0, 0) + 4L * ni.H * ni.W * 16 <
                                 (1L << 31) &&
                             im2col_lds_bytes(st.cs) <= kIm2colMaxLds && ni.N <= 65535 && ni.H <= 65535;
                    if (st.i2c) {
                        // KCRS -> K(RS)C: channel (r * S + s) * C + c of the 1x1 filter
                        std::vector<float> wt(w.size());
                        for (long k = 0; k < d.K; ++k)
                            for (int c = 0; c < C; ++c)
                                for (int rs = 0; rs < d.R * d.S; ++rs)
                                    wt[(k * d.R * d.S + rs) * C + c] = w[(k * C + c) * d.R * d.S + rs];
                        w.swap(wt);
                    }
                    st.kcrs_off = add_params(P, w);
                    st.ws8_off = add_params(P, std::vector<float>((size_t)cdiv(d.K, 16) * 16, 1.f));
                    auto take = [&](long bytes) {
                        const long off = P->i8_bytes;
                        P->i8_bytes += (bytes + 255) / 256 * 256;
                        return off;
                    };
                    const ConvShape s8 = int8_conv_shape(st);
                    st.w8_off = take((long)int8_filter_bytes(s8.K, s8.C, s8.R, s8.S));
                    st.c8 = choose_int8_config(s8);
                }
                st.cc = choose_conv_config(st.cs);
                if (!(P->flags & NEO_PLAN_HOST_ONLY)) st.tuned = tuned_config(st.cs, true, &st.cc);
                const int v = B.new_val(id, ni.N, ni.C, ni.H, ni.W, ni.oc);
                st.out = v;
                P->steps.push_back(st);
                B.produce(id, v);
                break;
            }
            case NEO_OP_MAXPOOL:
            case NEO_OP_AVGPOOL: {
                const int lay = arriving(0) ? arriving(0) : D;
                Step st{};
                st.kind = d.op == NEO_OP_MAXPOOL ? ST_MAXPOOL : ST_AVGPOOL;
                st.node = id;
                st.in = B.get(ni.inputs[0], lay, id);
                st.ps = PoolShape{ni.N, ni.C, a->H, a->W, d.R, d.S, d.stride_h, d.stride_w,
                                  d.pad_h, d.pad_w, ni.H, ni.W, 0, cdiv(ni.C, lay)};
                st.ps.xb = lay;
                const int v = B.new_val(id, ni.N, ni.C, ni.H, ni.W, lay);
                st.out = v;
                P->steps.push_back(st);
                B.produce(id, v);
                break;
            }
            case NEO_OP_GAP: {
                const int lay = arriving(0) ? arriving(0) : D;
                Step st{};
                st.kind = ST_GAP;
                st.node = id;
                st.in = B.get(ni.inputs[0], lay, id);
                const int v = B.new_val(id, ni.N, ni.C, 1, 1, lay);
                st.out = v;
                P->steps.push_back(st);
                B.produce(id, v);
                break;
            }
            case NEO_OP_CONCAT: {
                auto whole = [&](int L) {
                    for (int j : ni.inputs)
                        if (P->nodes[j].C % L) return false;
                    return true;
                };
                int layout = 0;
                if (!naive) {
                    if (arriving(0) > 0 && whole(arriving(0)))
                        layout = arriving(0);
                    else if (whole(D))
                        layout = D;
                }
                for (size_t j = 0; j < ni.inputs.size(); ++j) B.get(ni.inputs[j], layout, id);
                const int v = B.new_val(id, ni.N, ni.C, ni.H, ni.W, layout);
                B.versions[id][layout] = v;
                ni.val = v;
                break;
            }
            case NEO_OP_FLATTEN: {
                const int src = B.get(ni.inputs[0], 0, id);
                const int v = B.new_val(id, ni.N, ni.C, 1, 1, 0);
                P->vals[v].alias_of = src;
                B.versions[id][0] = v;
                ni.val = v;
                break;
            }
            case NEO_OP_DENSE: {
                Step st{};
                st.kind = ST_DENSE;
                st.node = id;
                st.in = B.get(ni.inputs[0], 0, id);
                st.dense_in = a->C;
                st.dense_out = d.K;
                st.act = d.act;
                std::vector<float> w(d.w, d.w + (long)d.K * a->C);
                st.w_off = add_params(P, w);
                if (d.bias) st.b_off = add_params(P, std::vector<float>(d.bias, d.bias + d.K));
                if (P->flags & NEO_PLAN_INT8) {
                    // integer dense layer: int8 rows and their scales (packed on the device)
                    if ((long)a->C * 127 * 127 >= (1L << 31) ||
                        (long)d.K * (long)dense_i8_row_bytes(a->C) >= (1L << 31))
                        return fail(NEO_ERR_UNSUPPORTED, where + "int8 dense layer too wide for int32 sums "
                                                                 "or 2 GiB of weights");
                    st.i8 = true;
                    // from 8 images on, a 1x1 conv over a 1x1 map: the conv
                    // kernel's int8 input [N][ceil(IN/16)][1][1][16] is these
                    // rows, and its float32 output [N][OUT/16][1][1][16] the
                    // plain [N][OUT] when OUT is a multiple of 16
                    st.d_conv = ni.N >= 8 && d.K % 16 == 0 && (long)a->C <= 133000;
                    st.ws8_off = add_params(P, std::vector<float>((size_t)cdiv(d.K, 16) * 16, 1.f));
                    st.w8_off = P->i8_bytes;
                    const long wbytes = st.d_conv ? (long)int8_filter_bytes(d.K, a->C, 1, 1)
                                                  : (long)d.K * (long)dense_i8_row_bytes(a->C);
                    P->i8_bytes += (wbytes + 255) / 256 * 256;
                    if (st.d_conv) {
                        st.cs = ConvShape{ni.N, a->C, 1, 1, d.K, 1, 1, 1, 1, 0, 0, 1, 1, 0, d.K / 16, d.act};
                        st.c8 = choose_int8_config(st.cs);
                    }
                }
                const int v = B.new_val(id, ni.N, ni.C, 1, 1, 0);
                st.out = v;
                P->steps.push_back(st);
                B.produce(id, v);
                break;
            }
            case NEO_OP_OUTPUT: {
                const int src = B.get(ni.inputs[0], 0, id);
                P->out_val = src;
                ni.val = src;
                P->out_dims[0] = ni.N; P->out_dims[1] = ni.C; P->out_dims[2] = ni.H; P->out_dims[3] = ni.W;
                break;
            }
        }
    }

    // ---- consumer counts (a concat input may have no other reader) --------------------
    for (const Step& st : P->steps) {
        if (st.in >= 0) P->vals[st.in].consumers++;
        if (st.res >= 0) P->vals[st.res].consumers++;
    }
    for (auto& v : P->vals)
        if (v.alias_of >= 0) P->vals[v.alias_of].consumers++;
    P->vals[P->out_val].consumers++;
    for (int id : P->order) {
        const NodeInfo& ni = P->nodes[id];
        if (ni.nd.op != NEO_OP_CONCAT) continue;
        const int layout = P->vals[ni.val].layout;
        for (int j : ni.inputs) P->vals[B.versions[j][layout]].consumers++;
    }

    // ---- storage: concat views (outermost concat first), then own buffers ------------
    for (auto it = P->order.rbegin(); it != P->order.rend(); ++it) {
        const NodeInfo& ni = P->nodes[*it];
        if (ni.nd.op != NEO_OP_CONCAT) continue;
        Val& cv = P->vals[ni.val];
        if (!cv.view) {
            cv.c_off = 0;
            cv.c_tot = units(cv.C, cv.layout);
        }
        int off = cv.c_off;
        for (int j : ni.inputs) {
            const int u = B.versions[j][cv.layout];
            Val& uv = P->vals[u];
            if (uv.buf == kExtIn || uv.alias_of >= 0 || uv.view || uv.consumers != 1)
                return fail(NEO_ERR_UNSUPPORTED,
                            "concat node " + std::to_string(*it) + ": input " + std::to_string(j) +
                                " is read elsewhere or is the network input (no in-place slice)");
            uv.view = true;
            uv.c_off = off;
            uv.c_tot = cv.c_tot;
            uv.buf = -3 - ni.val;  // resolved below to the concat value's root
            off += units(uv.C, cv.layout);
        }
    }
    // own buffers for roots
    for (size_t i = 0; i < P->vals.size(); ++i) {
        Val& v = P->vals[i];
        if (v.alias_of >= 0 || v.buf == kExtIn || v.view) continue;
        v.buf = (int)P->buf_bytes.size();
        v.c_off = 0;
        v.c_tot = units(v.C, v.layout);
        P->buf_bytes.push_back(val_elems_root(v) * 4);
    }
    // resolve views (a view's concat value may itself be a view: walk outward)
    for (size_t i = 0; i < P->vals.size(); ++i) {
        Val& v = P->vals[i];
        int b = v.buf;
        while (b <= -3) b = P->vals[-3 - b].buf;
        v.buf = b;
    }
    // aliases share their source's storage (units converted if the layout
    // differs; only 1x1 maps whose channel count both blocks divide are
    // aliased, where the two layouts coincide)
    for (size_t i = 0; i < P->vals.size(); ++i) {
        Val& v = P->vals[i];
        if (v.alias_of < 0) continue;
        int r = v.alias_of;
        while (P->vals[r].alias_of >= 0) r = P->vals[r].alias_of;
        const Val& s = P->vals[r];
        v.buf = s.buf;
        v.view = s.view;
        const int f_s = s.layout ? s.layout : 1, f_v = v.layout ? v.layout : 1;
        v.c_off = s.c_off * f_s / f_v;
        v.c_tot = s.c_tot * f_s / f_v;
    }
    // the output goes straight into the caller's buffer when its storage is a
    // whole buffer of exactly the output's size; otherwise a copy step is added
    {
        const Val& o = P->vals[P->out_val];
        const long out_bytes = (long)o.N * o.C * o.H * o.W * 4;
        if (o.buf >= 0 && !o.view && P->buf_bytes[o.buf] == out_bytes) {
            P->ext_out_buf = o.buf;
        } else {
            Step st{};
            st.kind = ST_COPY;
            st.node = P->order.back();
            st.in = P->out_val;
            P->steps.push_back(st);
        }
    }
    long off = 0;
    for (long b : P->buf_bytes) {
        P->buf_off.push_back(off);
        off += align_up(b, 256);
    }
    P->act_bytes = off;
    // step output views
    for (Step& st : P->steps) {
        if (st.kind == ST_CONV) {
            st.cs.y_off = P->vals[st.out].c_off;
            st.cs.y_tot = P->vals[st.out].c_tot;
        } else if (st.kind == ST_MAXPOOL || st.kind == ST_AVGPOOL) {
            st.ps.y_off = P->vals[st.out].c_off;
            st.ps.y_tot = P->vals[st.out].c_tot;
        }
    }
    return NEO_OK;
}

// NEO_PLAN_GROUP: list scheduling of the steps.  Every value has storage of
// its own or a slice of a concatenation's, and none is reused, so a step has
// to wait only for the earlier steps that wrote storage it reads.  The steps
// are taken in rounds: each round holds every step whose producers ran in an
// earlier round; its NCHW16c convs of more than 4 input channels become
// launches of up to kMaxGroupConvs convs (in their original order), and each
// of its pooling steps rides along in one of those launches (in workgroups
// after the convs'; a lone conv becomes a one-conv launch for it); its other
// steps run one by one.  Steps of one round are independent, so one grid can
// run them all; at small batch sizes that fills the GPU where each alone
// would not, and saves launches.
void group_ready_convs(neo_plan* P) {
    std::vector<Step>& S = P->steps;
    const int n = (int)S.size();
    struct Extent {
        int buf;
        long lo, hi;  // channel range in the root buffer
    };
    auto extent = [&](int v) {
        const Val& x = P->vals[v];
        const long f = x.layout ? x.layout : 1;
        return Extent{x.buf, x.c_off * f, (x.c_off + units(x.C, x.layout)) * f};
    };
    auto overlap = [](const Extent& a, const Extent& b) {
        return a.buf == b.buf && a.buf != kExtIn && a.lo < b.hi && b.lo < a.hi;
    };
    std::vector<std::vector<int>> deps(n);
    for (int j = 0; j < n; ++j) {
        std::vector<Extent> reads;
        if (S[j].in >= 0) reads.push_back(extent(S[j].in));
        if (S[j].res >= 0) reads.push_back(extent(S[j].res));
        for (int i = 0; i < j; ++i) {
            bool dep = false;
            for (int o : {S[i].out, S[i].out2}) {
                if (o < 0) continue;
                const Extent w = extent(o);
                for (const Extent& r : reads) dep = dep || overlap(w, r);
            }
            if (dep) deps[j].push_back(i);
        }
    }
    // a pooling step of the round rides along in one of its conv launches
    // (NEO_GROUP_POOLS=0 keeps pools in launches of their own)
    const char* gp = std::getenv("NEO_GROUP_POOLS");
    const bool pools_ride = !(gp && gp[0] == '0');
    std::vector<char> done(n, 0);
    std::vector<Step> out;
    for (int left = n; left > 0;) {
        std::vector<int> ready, convs, pools;
        for (int j = 0; j < n; ++j) {
            if (done[j]) continue;
            bool ok = true;
            for (int d : deps[j]) ok = ok && done[d];
            if (ok) ready.push_back(j);
        }
        for (int j : ready) {
            if (S[j].kind == ST_CONV && (S[j].i8 || conv_group_eligible(S[j].cs)))
                convs.push_back(j);
            else if (pools_ride && (S[j].kind == ST_MAXPOOL || S[j].kind == ST_AVGPOOL) && S[j].p8 < 0)
                pools.push_back(j);
            else
                out.push_back(S[j]);
        }
        size_t next_pool = 0;
        for (size_t k = 0; k < convs.size(); k += kMaxGroupConvs) {
            const size_t e = std::min(convs.size(), k + kMaxGroupConvs);
            const bool with_pool = next_pool < pools.size();
            if (e - k == 1 && !with_pool) {
                out.push_back(S[convs[k]]);
                continue;
            }
            Step grp{};
            if (with_pool) grp.pools.push_back(S[pools[next_pool++]]);
            grp.kind = ST_CONV_GROUP;
            grp.node = S[convs[k]].node;
            grp.in = S[convs[k]].in;
            for (size_t m = k; m < e; ++m) grp.members.push_back(S[convs[m]]);
            std::vector<ConvShape> shp;
            for (const Step& m : grp.members) shp.push_back(m.i8 ? int8_conv_shape(m) : m.cs);
            if (grp.members[0].i8) {
                // integer convs (an int8 plan has no others): one int8
                // configuration for all members
                grp.i8 = true;
                grp.c8 = choose_int8_group_config(shp.data(), (int)shp.size());
                for (Step& m : grp.members) {
                    m.c8 = grp.c8;
                    m.tuned = false;
                }
                out.push_back(grp);
                continue;
            }
            grp.cc = choose_group_config(shp.data(), (int)shp.size());
            // launch-configuration sweeps: "fk,fp,waves" for every group it suits
            if (const char* ev = std::getenv("NEO_GROUP_CONFIG")) {
                ConvConfig t{1, 1, 1, 1};
                if (std::sscanf(ev, "%d,%d,%d", &t.fk, &t.fp, &t.waves) == 3 &&
                    conv_group_config_valid(shp.data(), (int)shp.size(), t)) {
                    grp.cc = t;
                    grp.tuned = true;  // kept as given, not searched
                }
            }
            for (Step& m : grp.members) m.cc = grp.cc;
            out.push_back(grp);
        }
        for (; next_pool < pools.size(); ++next_pool) out.push_back(S[pools[next_pool]]);
        for (int j : ready) done[j] = 1;
        left -= (int)ready.size();
    }
    S.swap(out);
}

// NEO_PLAN_FUSE_GAP: a global average pool whose input is one image's output
// of a conv step (read by nothing else) and whose result only dense layers
// read (through a flatten, and the transform to NCHW before it) is folded
// into both: the conv writes, instead of
// its outputs, the channel sums of every 16 pixels, and each dense layer
// reads their mean.  One launch less, and the conv's output never goes to
// memory.
void fuse_gap(neo_plan* P) {
    std::vector<Step>& S = P->steps;
    auto root = [&](int v) {
        while (P->vals[v].alias_of >= 0) v = P->vals[v].alias_of;
        return v;
    };
    std::vector<char> drop(S.size(), 0);
    for (size_t j = 0; j < S.size(); ++j) {
        if (S[j].kind != ST_GAP) continue;
        const int in = S[j].in, g = S[j].out;
        const Val& iv = P->vals[in];
        // (the dense layer sums the input's rows in 64 KB of LDS)
        if (iv.N != 1 || iv.view || iv.alias_of >= 0 || iv.consumers != 1 || iv.C % 4 || iv.C > 16384)
            continue;
        int pi = -1;
        for (size_t i = 0; i < j; ++i)
            if (S[i].out == in) pi = (int)i;
        if (pi < 0 || S[pi].kind != ST_CONV) continue;
        // the pooled value and its transforms (a 1x1 map: to NCHW for the
        // flatten); every reader must be a dense layer or such a transform
        std::vector<int> pooled{g};
        auto is_pooled = [&](int v) {
            return v >= 0 && std::find(pooled.begin(), pooled.end(), root(v)) != pooled.end();
        };
        std::vector<size_t> dense, xforms;
        bool ok = true;
        for (size_t k = j + 1; k < S.size() && ok; ++k) {
            if (is_pooled(S[k].res)) ok = false;
            if (!is_pooled(S[k].in)) continue;
            if (S[k].kind == ST_TRANSFORM) {
                pooled.push_back(S[k].out);
                xforms.push_back(k);
            } else if (S[k].kind == ST_DENSE && S[k].dense_in == iv.C) {
                dense.push_back(k);
            } else {
                ok = false;
            }
        }
        ok = ok && !is_pooled(P->out_val);
        for (size_t v = 0; v < P->vals.size(); ++v) ok = ok && !(P->vals[v].view && is_pooled((int)v));
        if (!ok || dense.empty()) continue;
        S[pi].cs.gap = 1;
        // the streaming pointwise kernel has no folded pool: the tile kernel's
        // configuration for this shape instead
        if (S[pi].cc.fp == 0) S[pi].cc = choose_conv_config(S[pi].cs);
        const int hw = iv.H * iv.W;
        for (size_t k : dense) {
            S[k].in = in;  // reads the conv's sums (and so runs after it)
            S[k].gap_parts = cdiv(hw, 16);
            S[k].gap_stride = cdiv(iv.C, 16) * 16;
            S[k].gap_scale = 1.f / (float)hw;
        }
        drop[j] = 1;
        for (size_t k : xforms) drop[k] = 1;
    }
    std::vector<Step> out;
    for (size_t j = 0; j < S.size(); ++j)
        if (!drop[j]) out.push_back(S[j]);
    S.swap(out);
}

// NEO_PLAN_FUSE_PAIRS: a pointwise conv whose output is the input of a later
// pointwise conv with a kernel for the pair (conv_pair_eligible) runs with it
// in one launch, at the first conv's place (the second reads nothing else, so
// its inputs are ready there).  The first output is still stored; other
// readers keep reading it.  Tuning splits a pair that measures slower than
// its two convs alone.
void fuse_pairs(neo_plan* P) {
    std::vector<Step>& S = P->steps;
    std::vector<char> taken(S.size(), 0);
    std::vector<Step> out;
    for (size_t i = 0; i < S.size(); ++i) {
        if (taken[i]) continue;
        bool paired = false;
        for (size_t j = i + 1; j < S.size() && S[i].kind == ST_CONV && !paired; ++j) {
            const Step& b = S[j];
            if (taken[j] || b.kind != ST_CONV || b.in != S[i].out || b.res >= 0 ||
                P->vals[S[i].out].view || !conv_pair_eligible(S[i].cs, b.cs))
                continue;
            Step pr{};
            pr.kind = ST_CONV_PAIR;
            pr.node = S[i].node;
            pr.in = S[i].in;
            pr.res = S[i].res;
            pr.out = S[i].out;
            pr.out2 = b.out;
            pr.members = {S[i], b};
            taken[j] = 1;
            out.push_back(pr);
            paired = true;
        }
        if (!paired) out.push_back(S[i]);
    }
    S.swap(out);
}

// NEO_PLAN_FUSE_CHAINS: a 3x3 conv whose output only a pointwise conv reads
// (alone, or as the first of a pair) runs with it in one launch where a
// kernel exists for the channel counts (conv_chain_eligible), at the
// pointwise step's place; the 3x3's output is then never stored.  Tuning
// splits a chain that measures slower than its parts.
void fuse_chains(neo_plan* P) {
    std::vector<Step>& S = P->steps;
    std::vector<char> drop(S.size(), 0);
    for (size_t j = 0; j < S.size(); ++j) {
        Step& X = S[j];
        std::vector<Step> tail;
        if (X.kind == ST_CONV_PAIR)
            tail = X.members;
        else if (X.kind == ST_CONV)
            tail = {X};
        else
            continue;
        const int v = tail[0].in;
        const Val& mv = P->vals[v];
        if (mv.buf == kExtIn || mv.view || mv.alias_of >= 0 || mv.consumers != 1) continue;
        for (size_t i = 0; i < j; ++i) {
            if (drop[i] || S[i].kind != ST_CONV || S[i].out != v || S[i].res >= 0) continue;
            ConvShape shp[3];
            shp[0] = S[i].cs;
            for (size_t m = 0; m < tail.size(); ++m) shp[m + 1] = tail[m].cs;
            const int n = 1 + (int)tail.size();
            if (!conv_chain_eligible(shp, n)) break;
            Step ch{};
            ch.kind = ST_CONV_CHAIN;
            ch.node = S[i].node;
            ch.in = S[i].in;
            ch.res = tail[0].res;
            ch.out = tail[0].out;
            ch.out2 = n == 3 ? tail[1].out : -1;
            ch.members = {S[i]};
            ch.members.insert(ch.members.end(), tail.begin(), tail.end());
            X = ch;
            drop[i] = 1;
            break;
        }
    }
    std::vector<Step> out;
    for (size_t j = 0; j < S.size(); ++j)
        if (!drop[j]) out.push_back(S[j]);
    S.swap(out);
}

// NEO_PLAN_FUSE_POOL: a small-channel conv (a network stem) whose output
// only a max pooling step reads runs with it in one launch (conv_pool.hip),
// at the conv's place; the conv's output is then never stored.  Tuning
// splits the pair back where the two launches measure faster.
void fuse_conv_pool(neo_plan* P) {
    std::vector<Step>& S = P->steps;
    std::vector<char> drop(S.size(), 0);
    for (size_t i = 0; i < S.size(); ++i) {
        Step& c = S[i];
        if (c.kind != ST_CONV || c.res >= 0) continue;
        const Val& mv = P->vals[c.out];
        if (mv.buf == kExtIn || mv.buf == P->ext_out_buf || mv.view || mv.alias_of >= 0 ||
            mv.consumers != 1)
            continue;
        for (size_t j = i + 1; j < S.size(); ++j) {
            if (S[j].kind != ST_MAXPOOL || S[j].in != c.out) continue;
            if (!conv_pool_eligible(c.cs, S[j].ps)) break;
            Step f{};
            f.kind = ST_CONV_POOL;
            f.node = c.node;
            f.in = c.in;
            f.out = S[j].out;
            f.members = {c};
            f.pools = {S[j]};
            f.cpc = choose_conv_pool_config(c.cs, S[j].ps);
            // launch-configuration override "fk,fp,waves,ty,tx" (tests and sweeps)
            if (const char* ev = std::getenv("NEO_CONVPOOL_CONFIG")) {
                ConvPoolConfig k{};
                if (std::sscanf(ev, "%d,%d,%d,%d,%d", &k.fk, &k.fp, &k.waves, &k.ty, &k.tx) == 5 &&
                    conv_pool_config_valid(c.cs, S[j].ps, k))
                    f.cpc = k;
            }
            c = f;
            drop[j] = 1;
            break;
        }
    }
    std::vector<Step> out;
    for (size_t j = 0; j < S.size(); ++j)
        if (!drop[j]) out.push_back(S[j]);
    S.swap(out);
}

float* val_ptr(const neo_plan* P, int v, const float* x_in, float* y_out) {
    const Val& val = P->vals[v];
    if (val.buf == kExtIn) return const_cast<float*>(x_in);
    if (val.buf == P->ext_out_buf) return y_out;
    return reinterpret_cast<float*>(P->d_act + P->buf_off[val.buf]);
}

// The pooling step riding in a fused conv launch, with its buffers.
bool group_pool(const neo_plan* P, const Step& s, const float* x_in, float* y_out, GroupPool* gp) {
    if (s.pools.empty()) return false;
    const Step& ps = s.pools[0];
    gp->s = ps.ps;
    gp->max = ps.kind == ST_MAXPOOL;
    gp->x = val_ptr(P, ps.in, x_in, y_out);
    gp->y = val_ptr(P, ps.out, x_in, y_out);
    gp->q = PoolQ{};
    if (ps.q_out >= 0 && !P->i8_f32_out) {
        // NEO_PLAN_INT8: the int8 copy its conv readers share
        const I8Copy& qo = P->i8_copies[ps.q_out];
        gp->q.yq = P->d_i8 + qo.xq_off;
        gp->q.scale = qo.xscale;
        gp->q.qph = qo.ph;
        gp->q.qpw = qo.pw;
        gp->q.q_off = ps.q_off8 >= 0 ? ps.q_off8 : 0;
        gp->q.q_tot = ps.q_tot8 > 0 ? ps.q_tot8 : 0;
        if (!ps.f32_needed) gp->y = nullptr;
    }
    return true;
}

// NEO_PLAN_INT8: one int8 copy per value that int8 convs read, shared by
// all of them (one scale: the value's), its halo the largest padding among
// them (each conv starts its windows that much further in).  The step
// producing the value writes the copy when it is a conv (requantizing its
// epilogue's value) or a pooling step (quantizing its output), beside its
// float32 output if anything else reads that; otherwise the first conv to
// read the copy runs its quantization pass.
void plan_int8_copies(neo_plan* P) {
    const int ns = (int)P->steps.size();
    // the value itself, through aliases (a flatten reads its source's storage)
    auto root = [&](int v) {
        while (P->vals[v].alias_of >= 0) v = P->vals[v].alias_of;
        return v;
    };
    for (int i = 0; i < ns; ++i) {
        Step& t = P->steps[i];
        if (!((t.kind == ST_CONV || t.kind == ST_DENSE) && t.i8)) continue;
        const bool rows = t.kind == ST_DENSE;
        int c = -1;
        for (int k = 0; k < (int)P->i8_copies.size() && !t.i2c; ++k)
            if (P->i8_copies[k].val == t.in && P->i8_copies[k].rows == rows && !P->i8_copies[k].im2col) c = k;
        if (c < 0) {
            c = (int)P->i8_copies.size();
            I8Copy q{t.in, rows || t.i2c ? 0 : t.cs.ph, rows || t.i2c ? 0 : t.cs.pw, -1};
            q.rows = rows;
            q.im2col = t.i2c;
            q.ics = t.cs;
            P->i8_copies.push_back(q);
            t.quant_here = true;  // the first reader, unless a writer takes it over
        }
        I8Copy& q = P->i8_copies[c];
        if (!rows && !t.i2c) {
            q.ph = std::max(q.ph, t.cs.ph);
            q.pw = std::max(q.pw, t.cs.pw);
        }
        t.qc = c;
    }
    for (I8Copy& q : P->i8_copies) {
        const Val& v = P->vals[q.val];
        q.xq_off = P->i8_bytes;
        const ConvShape is = im2col_shape(q.ics);
        const long bytes = q.rows     ? (long)v.N * (long)dense_i8_row_bytes(v.C * v.H * v.W)
                           : q.im2col ? (long)int8_act_bytes(is.N, is.C, is.H, is.W, 0, 0)
                                      : (long)int8_act_bytes(v.N, v.C, v.H, v.W, q.ph, q.pw);
        P->i8_bytes += (bytes + 255) / 256 * 256;
    }
    for (int c = 0; c < (int)P->i8_copies.size(); ++c) {
        I8Copy& q = P->i8_copies[c];
        if (q.im2col) continue;  // its conv's own pass
        int w = -1;
        for (int i = 0; i < ns; ++i) {
            const Step& t = P->steps[i];
            // a conv or pool writes a conv input's copy; a dense layer the next dense layer's
            // a dense layer's rows: the dense layer before it, the global pool
            // (NCHW16c, whole blocks: its means are the rows) or the exit of
            // the blocked layout (NCHW16c -> NCHW, not into a slice)
            const Val* to = t.out >= 0 ? &P->vals[t.out] : nullptr;
            const bool kind_ok =
                q.rows ? ((t.kind == ST_DENSE && t.i8) ||
                          (t.kind == ST_GAP && to->layout == 16 && to->C % 16 == 0) ||
                          (t.kind == ST_TRANSFORM && t.src_block == 16 && t.dst_block == 0 && !to->view &&
                           to->alias_of < 0 && !P->vals[t.in].view))
                       : ((t.kind == ST_CONV && t.i8) || t.kind == ST_MAXPOOL || t.kind == ST_AVGPOOL);
            if (t.out >= 0 && root(t.out) == root(q.val) && kind_ok) w = i;
        }
        if (w < 0) continue;
        // the writer: does anything other than this copy's int8 readers read
        // its float32 output (itself or an alias of it: a flatten), or is
        // it the network's output or a concatenation's slice?
        const int rv = root(q.val);
        auto same = [&](int v) { return v >= 0 && root(v) == rv; };
        bool f32 = false;
        for (int o = 0; o < (int)P->vals.size(); ++o)
            if (same(o) && (o == P->out_val || P->vals[o].view)) f32 = true;
        for (int i = 0; i < ns; ++i) {
            const Step& t = P->steps[i];
            const bool int8_reader = (t.kind == ST_CONV || t.kind == ST_DENSE) && t.i8 && t.qc == c;
            if ((same(t.in) && !int8_reader) || same(t.res) || (t.out2 >= 0 && same(t.out2))) f32 = true;
            for (const Step& m : t.members)
                if (same(m.in) || same(m.res)) f32 = true;
        }
        q.writer = w;
        P->steps[w].q_out = c;
        P->steps[w].f32_needed = f32;
        for (Step& t : P->steps)
            if (t.qc == c) t.quant_here = false;
    }
    // a concatenation (nothing produces it as a whole) whose parts are all
    // produced by int8 convs or pooling steps: each part's producer writes
    // its slice of the copy, with the concatenation's scale
    for (int c = 0; c < (int)P->i8_copies.size(); ++c) {
        I8Copy& q = P->i8_copies[c];
        const Val& cv = P->vals[q.val];
        if (q.writer >= 0 || q.im2col || cv.node < 0 || P->nodes[cv.node].nd.op != NEO_OP_CONCAT ||
            cv.layout != 16 || cv.view)
            continue;
        std::vector<std::pair<int, int>> parts;  // (producer step, block offset in the concatenation)
        // the parts of concatenation node `node`, through nested
        // concatenations (views whose offsets are in the root buffer)
        std::function<bool(int)> collect = [&](int node) {
            for (int j : P->nodes[node].inputs) {
                int u = -1;
                for (int k = 0; k < (int)P->vals.size(); ++k)
                    if (P->vals[k].node == j && P->vals[k].view && P->vals[k].layout == cv.layout &&
                        P->vals[k].alias_of < 0)
                        u = k;
                if (u < 0) return false;
                if (P->nodes[j].nd.op == NEO_OP_CONCAT) {
                    if (!collect(j)) return false;
                    continue;
                }
                int w = -1;
                for (int i = 0; i < ns; ++i) {
                    const Step& t = P->steps[i];
                    if (t.out == u && ((t.kind == ST_CONV && t.i8) || t.kind == ST_MAXPOOL || t.kind == ST_AVGPOOL))
                        w = i;
                }
                if (w < 0 || P->steps[w].q_out >= 0) return false;
                parts.emplace_back(w, P->vals[u].c_off - cv.c_off);
            }
            return true;
        };
        if (!collect(cv.node) || parts.empty()) continue;
        bool f32 = q.val == P->out_val || cv.view;
        for (const Val& o : P->vals)
            if (o.alias_of == q.val) f32 = true;
        for (int i = 0; i < ns; ++i) {
            const Step& t = P->steps[i];
            if ((t.in == q.val && !(t.kind == ST_CONV && t.i8 && !t.i2c)) || t.res == q.val) f32 = true;
        }
        q.assembled = true;
        for (const auto& pw : parts) {
            Step& t = P->steps[pw.first];
            t.q_out = c;
            t.f32_needed = f32;
            t.q_off8 = pw.second;
            t.q_tot8 = cdiv(cv.C, 16);
        }
        for (Step& t : P->steps)
            if (t.qc == c) t.quant_here = false;
    }
}

// NEO_PLAN_INT8: an im2col copy whose value is only the NCHW -> NCHW16c
// transform of a plain NCHW value (a network's input) read by nothing else:
// the pass reads the NCHW value and the transform step goes (at batch 32 it
// would write 16 float lanes per pixel for 3 channels).
void drop_im2col_transforms(neo_plan* P) {
    for (I8Copy& q : P->i8_copies) {
        if (!q.im2col) continue;
        int ti = -1, readers = 0;
        for (int i = 0; i < (int)P->steps.size(); ++i) {
            const Step& t = P->steps[i];
            if (t.kind == ST_TRANSFORM && t.out == q.val && t.src_block == 0 && t.dst_block == 16) ti = i;
            if (t.in == q.val || t.res == q.val || t.out2 == q.val) ++readers;
            for (const Step& m : t.members)
                if (m.in == q.val || m.res == q.val) ++readers;
        }
        bool plain = q.val != P->out_val && !P->vals[q.val].view;
        for (const Val& v : P->vals)
            if (v.alias_of == q.val) plain = false;
        if (ti < 0 || readers != 1 || !plain) continue;
        const Val& sv = P->vals[P->steps[ti].in];
        if (sv.layout != 0 || sv.view || sv.alias_of >= 0) continue;
        q.src = P->steps[ti].in;
        P->steps.erase(P->steps.begin() + ti);
        for (I8Copy& o : P->i8_copies)
            if (o.writer > ti) --o.writer;
    }
}

// NEO_PLAN_INT8: a max pool that writes its output's int8 copy (int8 only)
// from a conv output nothing else reads pools that conv's output in int8
// instead: the conv requantizes by division with the pool copy's scale (no
// float32 output) and the pool takes byte maxima -- quantization by division
// is monotone, so these are the quantized maxima, the same bits.  Taken
// where the conv's float32 output is at least 16 MiB (measured: at batch 32
// the pool reads a quarter of the bytes and the conv writes a quarter; on
// batch-1 maps the dividing epilogue and the extra launch shape cost more
// than the bytes saved).
void int8_pool_inputs(neo_plan* P) {
    const int ns = (int)P->steps.size();
    for (int pi = 0; pi < ns; ++pi) {
        Step& p = P->steps[pi];
        if (p.kind != ST_MAXPOOL || p.q_out < 0 || p.f32_needed || p.q_off8 >= 0) continue;
        const int v = p.in;
        const Val& vv = P->vals[v];
        if (v == P->out_val || vv.view || vv.alias_of >= 0 || vv.layout != 16 ||
            (long)vv.N * cdiv(vv.C, 16) * 16 * vv.H * vv.W * 4 < (16L << 20))
            continue;
        int ci = -1, readers = 0;
        for (int i = 0; i < ns; ++i) {
            const Step& t = P->steps[i];
            if (t.out == v && t.kind == ST_CONV && t.i8 && t.q_out < 0) ci = i;
            if (t.in == v || t.res == v || t.out2 == v) ++readers;
        }
        for (const Val& o : P->vals)
            if (o.alias_of == v) ++readers;
        if (ci < 0 || readers != 1) continue;
        I8Copy q{v, 0, 0, P->i8_bytes};
        q.divide = true;
        q.pool_copy = p.q_out;
        q.writer = ci;
        P->i8_bytes += ((long)int8_act_bytes(vv.N, vv.C, vv.H, vv.W, 0, 0) + 255) / 256 * 256;
        P->i8_copies.push_back(q);
        P->steps[ci].q_out = (int)P->i8_copies.size() - 1;
        P->steps[ci].f32_needed = false;
        p.p8 = P->steps[ci].q_out;
    }
}

// NEO_PLAN_INT8 with NEO_PLAN_GROUP: grouping reorders the steps, so the
// quantization pass of a copy that no conv writes moves to the copy's first
// reader in the new order (a group runs its members' passes before its
// launch, so readers in the same launch see the copy complete).
void place_int8_quant_passes(neo_plan* P) {
    std::vector<char> seen(P->i8_copies.size(), 0);
    auto visit = [&](Step& t) {
        if (!((t.kind == ST_CONV || t.kind == ST_DENSE) && t.i8)) return;
        const I8Copy& q = P->i8_copies[t.qc];
        const bool first = q.writer < 0 && !q.assembled && !seen[t.qc];
        t.quant_here = first;
        seen[t.qc] = 1;
    };
    for (Step& t : P->steps) {
        visit(t);
        for (Step& m : t.members) visit(m);
    }
}

std::string describe(const neo_plan* P) {
    std::ostringstream o;
    auto lay = [](int l) { return l ? "NCHW" + std::to_string(l) + "c" : std::string("NCHW"); };
    o << "{\"input\":[" << P->N << "," << P->C << "," << P->H << "," << P->W << "],";
    o << "\"block\":" << P->block << ",\"naive\":" << ((P->flags & NEO_PLAN_NAIVE) ? "true" : "false");
    o << ",\"host_only\":" << ((P->flags & NEO_PLAN_HOST_ONLY) ? "true" : "false");
    o << ",\"hipgraph\":" << ((P->flags & NEO_PLAN_HIPGRAPH) ? "true" : "false");
    o << ",\"output\":[" << P->out_dims[0] << "," << P->out_dims[1] << "," << P->out_dims[2] << ","
      << P->out_dims[3] << "]";
    o << ",\"order\":[";
    for (size_t i = 0; i < P->order.size(); ++i) o << (i ? "," : "") << P->order[i];
    o << "],\"nodes\":[";
    for (size_t i = 0; i < P->nodes.size(); ++i) {
        const NodeInfo& ni = P->nodes[i];
        const Val& v = P->vals[ni.val];
        o << (i ? "," : "") << "{\"id\":" << i << ",\"op\":\"" << op_name(ni.nd.op)
          << "\",\"shape\":[" << ni.N << "," << ni.C << "," << ni.H << "," << ni.W
          << "],\"layout\":\"" << lay(v.layout) << "\",\"value\":" << ni.val << "}";
    }
    o << "],\"values\":[";
    for (size_t i = 0; i < P->vals.size(); ++i) {
        const Val& v = P->vals[i];
        o << (i ? "," : "") << "{\"id\":" << i << ",\"node\":" << v.node << ",\"layout\":\""
          << lay(v.layout) << "\",\"shape\":[" << v.N << "," << v.C << "," << v.H << "," << v.W
          << "],\"buf\":" << v.buf << ",\"c_off\":" << v.c_off << ",\"c_tot\":" << v.c_tot
          << ",\"view\":" << (v.view ? "true" : "false") << ",\"alias_of\":" << v.alias_of << "}";
    }
    o << "],\"transforms\":[";
    for (size_t i = 0; i < P->xforms.size(); ++i) {
        const Xform& x = P->xforms[i];
        o << (i ? "," : "") << "{\"from_value\":" << x.from_val << ",\"to_value\":" << x.to_val
          << ",\"from\":\"" << lay(x.from_layout) << "\",\"to\":\"" << lay(x.to_layout)
          << "\",\"before_node\":" << x.consumer_node << ",\"alias\":" << (x.alias ? "true" : "false")
          << "}";
    }
    o << "],\"n_transforms\":" << P->xforms.size() << ",\"steps\":[";
    static const char* kinds[] = {"transform", "conv", "maxpool", "avgpool", "gap", "dense", "copy",
                                  "conv_group", "conv_pair", "conv_chain", "conv_pool"};
    for (size_t i = 0; i < P->steps.size(); ++i) {
        const Step& s = P->steps[i];
        o << (i ? "," : "") << "{\"kind\":\"" << kinds[s.kind] << "\",\"node\":" << s.node
          << ",\"in\":" << s.in << ",\"out\":" << s.out << ",\"res\":" << s.res;
        auto conv_json = [&](const Step& s) {
            const ConvShape& c = s.cs;
            const ConvConfig& cfg = s.wino ? s.wc : s.cc;  // the configuration that runs
            o << "{\"N\":" << c.N << ",\"C\":" << c.C << ",\"H\":" << c.H << ",\"W\":" << c.W
              << ",\"K\":" << c.K << ",\"R\":" << c.R << ",\"S\":" << c.S << ",\"stride\":[" << c.sh
              << "," << c.sw << "],\"pad\":[" << c.ph << "," << c.pw << "],\"OH\":" << c.OH
              << ",\"OW\":" << c.OW << ",\"y_off\":" << c.y_off << ",\"y_tot\":" << c.y_tot
              << ",\"act\":" << c.act << ",\"bias\":" << (s.b_off >= 0 ? "true" : "false")
              << ",\"ic_bn\":" << c.xb << ",\"oc_bn\":" << c.yb
              << ",\"tile\":[" << cfg.fk << "," << cfg.fp << "],\"split\":" << cfg.split
              << ",\"waves\":" << cfg.waves << ",\"tuned\":" << (s.tuned ? "true" : "false")
              << ",\"algo\":\"" << (s.i8 ? "int8" : s.wino ? "winograd" : "direct") << "\"";
            if (s.i8) {
                char xs[32];
                std::snprintf(xs, sizeof xs, "%.9g", (double)P->i8_copies[s.qc].xscale);
                o << ",\"int8\":{\"tile\":[" << s.c8.fk << "," << s.c8.fp << "],\"waves\":" << s.c8.waves
                  << ",\"x_scale\":" << xs << ",\"calibrated\":" << (P->i8_ready ? "true" : "false")
                  << ",\"input_copy\":" << s.qc << ",\"quantizes_input\":"
                  << (s.quant_here ? "true" : "false") << ",\"writes_copy\":" << s.q_out
                  << ",\"writes_f32\":" << (s.f32_needed ? "true" : "false");
                if (s.i2c)
                    o << ",\"im2col\":" << (P->i8_copies[s.qc].src >= 0 ? "\"nchw\"" : "\"blocked\"");
                if (s.q_off8 >= 0) o << ",\"writes_slice\":[" << s.q_off8 << "," << s.q_tot8 << "]";
                o << "}";
            }
            if (c.gap) o << ",\"gap_sums\":true";
            o << "}";
        };
        if (s.kind == ST_CONV) {
            o << ",\"conv\":";
            conv_json(s);
        }
        if (s.kind == ST_CONV_GROUP) {
            const ConvConfig& gc = s.i8 ? s.c8 : s.cc;
            o << ",\"tile\":[" << gc.fk << "," << gc.fp << "],\"waves\":" << gc.waves
              << ",\"tuned\":" << (s.tuned ? "true" : "false") << ",\"algo\":\""
              << (s.i8 ? "int8" : "direct") << "\",\"members\":[";
            for (size_t m = 0; m < s.members.size(); ++m) {
                const Step& ms = s.members[m];
                o << (m ? "," : "") << "{\"node\":" << ms.node << ",\"in\":" << ms.in
                  << ",\"out\":" << ms.out << ",\"res\":" << ms.res << ",\"conv\":";
                conv_json(ms);
                o << "}";
            }
            o << "]";
            for (const Step& ps : s.pools) {
                o << ",\"pool\":{\"kind\":\"" << kinds[ps.kind] << "\",\"node\":" << ps.node
                  << ",\"in\":" << ps.in << ",\"out\":" << ps.out;
                if (ps.q_out >= 0) {
                    o << ",\"int8\":{\"writes_copy\":" << ps.q_out << ",\"writes_f32\":"
                      << (ps.f32_needed ? "true" : "false");
                    if (ps.q_off8 >= 0) o << ",\"writes_slice\":[" << ps.q_off8 << "," << ps.q_tot8 << "]";
                    o << "}";
                }
                o << "}";
            }
        }
        if (s.kind == ST_CONV_PAIR || s.kind == ST_CONV_CHAIN) {
            o << ",\"out2\":" << s.out2 << ",\"tuned\":" << (s.tuned ? "true" : "false") << ",\"members\":[";
            for (size_t m = 0; m < s.members.size(); ++m) {
                const Step& ms = s.members[m];
                o << (m ? "," : "") << "{\"node\":" << ms.node << ",\"in\":" << ms.in
                  << ",\"out\":" << ms.out << ",\"res\":" << ms.res << ",\"conv\":";
                conv_json(ms);
                o << "}";
            }
            o << "]";
        }
        if (s.kind == ST_CONV_POOL) {
            const Step& ms = s.members[0];
            const PoolShape& ps = s.pools[0].ps;
            o << ",\"tuned\":" << (s.tuned ? "true" : "false") << ",\"config\":{\"tile\":["
              << s.cpc.fk << "," << s.cpc.fp << "],\"waves\":" << s.cpc.waves << ",\"pooled_tile\":["
              << s.cpc.ty << "," << s.cpc.tx << "]},\"members\":[{\"node\":" << ms.node
              << ",\"in\":" << ms.in << ",\"out\":" << ms.out << ",\"res\":" << ms.res
              << ",\"conv\":";
            conv_json(ms);
            o << "}],\"pool\":{\"kind\":\"maxpool\",\"node\":" << s.pools[0].node
              << ",\"window\":[" << ps.R << "," << ps.S << "],\"stride\":[" << ps.sh << "," << ps.sw
              << "],\"pad\":[" << ps.ph << "," << ps.pw << "],\"OH\":" << ps.OH << ",\"OW\":" << ps.OW
              << "}";
        }
        if ((s.kind == ST_MAXPOOL || s.kind == ST_AVGPOOL || s.kind == ST_GAP || s.kind == ST_TRANSFORM) &&
            s.q_out >= 0) {
            o << ",\"int8\":{\"writes_copy\":" << s.q_out << ",\"writes_f32\":"
              << (s.f32_needed ? "true" : "false");
            if (s.q_off8 >= 0) o << ",\"writes_slice\":[" << s.q_off8 << "," << s.q_tot8 << "]";
            if (s.p8 >= 0) o << ",\"reads_int8\":" << s.p8;
            o << "}";
        }
        if (s.kind == ST_TRANSFORM) o << ",\"src_block\":" << s.src_block << ",\"dst_block\":" << s.dst_block;
        if (s.kind == ST_DENSE) {
            o << ",\"dense\":{\"in\":" << s.dense_in << ",\"out\":" << s.dense_out;
            if (s.gap_parts) o << ",\"gap_parts\":" << s.gap_parts;
            if (s.i8) {
                char xs[32];
                std::snprintf(xs, sizeof xs, "%.9g", (double)P->i8_copies[s.qc].xscale);
                o << ",\"algo\":\"int8\",\"int8\":{\"conv_mode\":" << (s.d_conv ? "true" : "false");
                if (s.d_conv)
                    o << ",\"tile\":[" << s.c8.fk << "," << s.c8.fp << "],\"waves\":" << s.c8.waves;
                o << ",\"x_scale\":" << xs << ",\"calibrated\":"
                  << (P->i8_ready ? "true" : "false") << ",\"input_copy\":" << s.qc
                  << ",\"quantizes_input\":" << (s.quant_here ? "true" : "false") << ",\"writes_copy\":"
                  << s.q_out << ",\"writes_f32\":" << (s.f32_needed ? "true" : "false") << "}";
            }
            o << "}";
        }
        o << "}";
    }
    o << "],\"buffers\":[";
    for (size_t i = 0; i < P->buf_bytes.size(); ++i) o << (i ? "," : "") << P->buf_bytes[i];
    o << "],\"activation_bytes\":" << P->act_bytes << ",\"param_bytes\":" << P->params.size() * 4
      << ",\"output_buffer\":" << P->ext_out_buf;
    if (P->searched)
        o << ",\"search\":{\"cost_us\":" << P->search_cost << ",\"fixed_block_cost_us\":"
          << P->fixed_cost << ",\"schemes_measured\":" << P->search_schemes
          << ",\"max_states\":" << P->search_states << "}";
    o << "}";
    return o.str();
}

// Candidate split factors of a channel count (Section 3.3.1: its factors) among
// the blocks the conv kernel implements, always with the plan's block; an
// input of at most 4 channels (the small-channel path) also takes 4.
std::vector<int> candidate_blocks(int C, int D, bool input_side) {
    std::vector<int> out;
    if (input_side && C <= 4) {  // the default layout (read as NCHW1c, no transform) or NCHW4c
        out.push_back(0);
        out.push_back(4);
    }
    for (int b : {16, 32, 64})
        if (b == D || (!(input_side && C <= 4) && C % b == 0 && b < C)) out.push_back(b);
    return out;
}

// NEO_PLAN_GLOBAL_SEARCH: measure every candidate scheme of every conv without
// a given scheme (the local search, its best launch configuration and time
// per (workload, ic_bn, oc_bn)) and every layout transform the program asks
// about, on zero-filled scratch buffers, then run the program and fix each
// conv's scheme.
int search_schemes(neo_plan* P) {
    hipError_t e;
    if (!P->cap_stream) {
        e = hipStreamCreateWithFlags(&P->cap_stream, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "neo_plan_create: search stream");
    }
    const hipStream_t st = P->cap_stream;
    long max_act = 0, max_w = 0, max_b = 16;
    for (const NodeInfo& ni : P->nodes) {
        max_act = std::max(max_act, (long)ni.N * cdiv(ni.C, 64) * 64 * ni.H * ni.W);
        if (ni.nd.op != NEO_OP_CONV) continue;
        const NodeInfo& a = P->nodes[ni.inputs[0]];
        ConvShape cs{};
        cs.C = a.C;
        cs.K = ni.nd.K;
        cs.R = ni.nd.R;
        cs.S = ni.nd.S;
        max_w = std::max(max_w, kernel_filter_floats(cs));
        max_b = std::max(max_b, (long)cdiv(ni.nd.K, 16) * 16);
    }
    float *X = nullptr, *Y = nullptr, *Rz = nullptr, *Wt = nullptr, *Bz = nullptr;
    e = hipMalloc(&X, max_act * 4);
    if (e == hipSuccess) e = hipMalloc(&Y, max_act * 4);
    if (e == hipSuccess) e = hipMalloc(&Rz, max_act * 4);
    if (e == hipSuccess) e = hipMalloc(&Wt, max_w * 4);
    if (e == hipSuccess) e = hipMalloc(&Bz, max_b * 4);
    for (auto* b : {X, Y, Rz})
        if (e == hipSuccess) e = hipMemset(b, 0, max_act * 4);
    if (e == hipSuccess) e = hipMemset(Wt, 0, max_w * 4);
    if (e == hipSuccess) e = hipMemset(Bz, 0, max_b * 4);
    int rc = e == hipSuccess ? NEO_OK : fail(NEO_ERR_OOM, "neo_plan_create: search buffers");
    // the first failed measurement (the program itself only sees an infinite time)
    int merr = NEO_OK;
    std::string merr_msg;
    auto measure_failed = [&](int code) {
        if (merr == NEO_OK) {
            merr = code;
            merr_msg = neo_last_error();
        }
    };

    const int D = P->block;
    Events ev;
    std::map<std::vector<int>, double> xmemo;
    std::map<std::vector<int>, double> cmemo;
    int measured = 0;
    auto conv_cost = [&](int v, int i, int j) -> double {
        const NodeInfo& ni = P->nodes[v];
        const int ib = kSearchBlocks[i], ob = kSearchBlocks[j];
        const NodeInfo& a = P->nodes[ni.inputs[0]];
        if (ni.ic) {  // the caller's scheme
            if (ib != read_layout(ni.ic) || ob != ni.oc) return INFINITY;
        } else {
            const std::vector<int> ci = candidate_blocks(a.C, D, true), co = candidate_blocks(ni.C, D, false);
            if (std::find(ci.begin(), ci.end(), ib) == ci.end() ||
                std::find(co.begin(), co.end(), ob) == co.end())
                return INFINITY;
        }
        const neo_node& d = ni.nd;
        ConvShape cs{ni.N, a.C, a.H, a.W, d.K, d.R, d.S, d.stride_h, d.stride_w, d.pad_h, d.pad_w,
                     ni.H, ni.W, 0, cdiv(d.K, ob), d.act};
        cs.xb = scheme_block(ib);
        cs.yb = ob;
        const bool has_res = d.residual >= 0, has_b = d.bn_gamma || d.bias;
        const std::vector<int> key{cs.N, cs.C, cs.H, cs.W, cs.K, cs.R, cs.S, cs.sh, cs.sw, cs.ph, cs.pw,
                                   ib, ob, has_res, has_b, cs.act};
        auto it = cmemo.find(key);
        if (it != cmemo.end()) return it->second;
        if (merr != NEO_OK) return INFINITY;
        ConvConfig cfg{};
        float us = 0.f;
        const int trc = tune_conv(cs, true, X, Wt, has_b ? Bz : nullptr, has_res ? Rz : nullptr, Y, st,
                                  &cfg, &us);
        if (trc != NEO_OK) measure_failed(trc);
        const double t = trc == NEO_OK ? us : INFINITY;
        ++measured;
        cmemo[key] = t;
        return t;
    };
    auto xform_cost = [&](int v, int i, int j) -> double {
        const NodeInfo& ni = P->nodes[v];
        const int sb = kSearchBlocks[i], db = kSearchBlocks[j];
        const std::vector<int> key{ni.N, ni.C, ni.H, ni.W, sb, db};
        auto it = xmemo.find(key);
        if (it != xmemo.end()) return it->second;
        if (merr != NEO_OK) return INFINITY;
        float us = 0.f;
        const hipError_t te = time_launch([&]() {
            return launch_layout_transform(X, sb, Y, db, ni.N, ni.C, ni.H, ni.W, 0, units(ni.C, db), st);
        }, st, ev.e0, ev.e1, &us);
        if (te != hipSuccess) measure_failed(hip_fail(te, "neo_plan_create: transform timing"));
        xmemo[key] = te != hipSuccess ? INFINITY : us;
        return xmemo[key];
    };
    std::vector<int> ic, oc;
    double best = 0, fixed = 0;
    long states = 0, fixed_states = 0;
    const std::vector<SearchNode> g = search_nodes(P);
    if (rc == NEO_OK)
        rc = layout_search_dp(g, P->order, D, conv_cost, xform_cost, &ic, &oc, &best, &states);
    if (rc == NEO_OK) {
        // the same program restricted to the plan's block everywhere (Section 3.2)
        std::vector<int> fi, fo;
        const int di = search_block_index(D);
        auto fixed_cost = [&](int v, int i, int j) -> double {
            if (P->nodes[v].ic) return conv_cost(v, i, j);
            return (i == di && j == di) ? conv_cost(v, i, j) : INFINITY;
        };
        rc = layout_search_dp(g, P->order, D, fixed_cost, xform_cost, &fi, &fo, &fixed, &fixed_states);
    }
    (void)hipStreamSynchronize(st);
    for (float* b : {X, Y, Rz, Wt, Bz})
        if (b) (void)hipFree(b);
    if (merr != NEO_OK) return fail(merr, merr_msg);
    if (rc != NEO_OK) return rc;
    for (size_t v = 0; v < P->nodes.size(); ++v) {
        NodeInfo& ni = P->nodes[v];
        if (ni.nd.op != NEO_OP_CONV || ni.ic) continue;
        ni.ic = scheme_block(ic[v]);
        ni.oc = oc[v];
    }
    P->searched = true;
    P->search_cost = best;
    P->fixed_cost = fixed;
    P->search_schemes = measured;
    P->search_states = states;
    return NEO_OK;
}

}  // namespace

extern "C" {

int neo_layout_search(const neo_node* nodes, int n_nodes, int N, int C, int H, int W, int block,
                      const double* conv_time, const double* xform_time, int* ic_bn, int* oc_bn,
                      double* cost) {
    if (!nodes || n_nodes <= 0 || !conv_time || !xform_time || !ic_bn || !oc_bn)
        return fail(NEO_ERR_INVALID_ARG, "neo_layout_search: NULL argument");
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0)
        return fail(NEO_ERR_INVALID_ARG, "neo_layout_search: non-positive input shape");
    if (block != 16 && block != 32 && block != 64)
        return fail(NEO_ERR_UNSUPPORTED, "neo_layout_search: block must be 16, 32 or 64");
    constexpr int NB = NEO_SEARCH_NB;
    try {
        neo_plan P;
        P.N = N; P.C = C; P.H = H; P.W = W; P.block = block;
        int rc = parse(&P, nodes, n_nodes, false);
        if (rc != NEO_OK) return rc;
        for (long i = 0; i < (long)n_nodes * NB * NB; ++i)
            if (!(xform_time[i] >= 0))
                return fail(NEO_ERR_INVALID_ARG, "neo_layout_search: transform times must be >= 0");
        auto conv_cost = [&](int v, int i, int j) -> double {
            const NodeInfo& ni = P.nodes[v];
            if (ni.ic && (kSearchBlocks[i] != read_layout(ni.ic) || kSearchBlocks[j] != ni.oc)) return INFINITY;
            const double t = conv_time[((long)v * NB + i) * NB + j];
            return (std::isfinite(t) && t >= 0) ? t : INFINITY;
        };
        auto xform_cost = [&](int v, int i, int j) { return xform_time[((long)v * NB + i) * NB + j]; };
        std::vector<int> ic, oc;
        double best = 0;
        long states = 0;
        rc = layout_search_dp(search_nodes(&P), P.order, block, conv_cost, xform_cost, &ic, &oc, &best,
                              &states);
        if (rc != NEO_OK) return rc;
        for (int v = 0; v < n_nodes; ++v) {
            ic_bn[v] = ic[v];
            oc_bn[v] = oc[v];
        }
        if (cost) *cost = best;
        return NEO_OK;
    } catch (const std::bad_alloc&) {
        return fail(NEO_ERR_OOM, "neo_layout_search: host allocation failed");
    }
}

int neo_plan_create(const neo_node* nodes, int n_nodes, int N, int C, int H, int W, int block,
                    unsigned flags, neo_plan** out) {
    if (!out) return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: out is NULL");
    *out = nullptr;
    if (!nodes || n_nodes <= 0) return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: no nodes");
    if (N <= 0 || C <= 0 || H <= 0 || W <= 0)
        return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: non-positive input shape");
    if (block != 16 && block != 32 && block != 64)
        return fail(NEO_ERR_UNSUPPORTED, "neo_plan_create: block must be 16, 32 or 64");
    if (flags & ~(unsigned)(NEO_PLAN_HOST_ONLY | NEO_PLAN_NAIVE | NEO_PLAN_HIPGRAPH | NEO_PLAN_TUNE |
                            NEO_PLAN_GLOBAL_SEARCH | NEO_PLAN_GROUP | NEO_PLAN_FUSE_GAP |
                            NEO_PLAN_FUSE_PAIRS | NEO_PLAN_FUSE_CHAINS | NEO_PLAN_FUSE_POOL |
                            NEO_PLAN_WINOGRAD | NEO_PLAN_INT8))
        return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: unknown flags");
    if ((flags & NEO_PLAN_INT8) &&
        ((flags & (NEO_PLAN_NAIVE | NEO_PLAN_GLOBAL_SEARCH | NEO_PLAN_FUSE_GAP |
                   NEO_PLAN_FUSE_PAIRS | NEO_PLAN_FUSE_CHAINS | NEO_PLAN_FUSE_POOL |
                   NEO_PLAN_WINOGRAD)) ||
         block != 16))
        return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: NEO_PLAN_INT8 plans its convs in NCHW16c "
                                         "(block 16; no naive transforms, search, fusion other "
                                         "than NEO_PLAN_GROUP, or Winograd)");
    if ((flags & (NEO_PLAN_TUNE | NEO_PLAN_GLOBAL_SEARCH)) && (flags & NEO_PLAN_HOST_ONLY))
        return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: tuning and search need a device plan");
    if ((flags & NEO_PLAN_GLOBAL_SEARCH) && (flags & NEO_PLAN_NAIVE))
        return fail(NEO_ERR_INVALID_ARG, "neo_plan_create: the global search plans without the naive transforms");
    if (flags & NEO_PLAN_GLOBAL_SEARCH) flags |= NEO_PLAN_TUNE;
    neo_plan* P = new (std::nothrow) neo_plan();
    if (!P) return fail(NEO_ERR_OOM, "neo_plan_create: host allocation failed");
    P->flags = flags;
    P->N = N; P->C = C; P->H = H; P->W = W; P->block = block;
    int rc;
    try {
        rc = parse(P, nodes, n_nodes, true);
        if (rc == NEO_OK && (flags & NEO_PLAN_GLOBAL_SEARCH)) rc = search_schemes(P);
        if (rc == NEO_OK) rc = build_steps(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_INT8)) {
            plan_int8_copies(P);
            drop_im2col_transforms(P);
            int8_pool_inputs(P);
            if (!(flags & NEO_PLAN_HOST_ONLY))
                for (Step& st : P->steps)
                    if ((st.kind == ST_CONV || (st.kind == ST_DENSE && st.d_conv)) && st.i8) {
                        const int mode = st.q_out < 0 ? 0 : st.f32_needed ? 3 : 2;
                        st.tuned = tuned_int8_config(int8_conv_shape(st), mode, &st.c8);
                    }
        }
        if (rc == NEO_OK && (flags & NEO_PLAN_FUSE_GAP)) fuse_gap(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_FUSE_PAIRS)) fuse_pairs(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_FUSE_CHAINS)) fuse_chains(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_FUSE_POOL)) fuse_conv_pool(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_GROUP)) group_ready_convs(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_GROUP) && (flags & NEO_PLAN_INT8)) place_int8_quant_passes(P);
        if (rc == NEO_OK && (flags & NEO_PLAN_WINOGRAD) && !(flags & NEO_PLAN_TUNE)) {
            // untuned, the convs still launched alone run the Winograd kernel
            // (with NEO_PLAN_TUNE the local search decides, conv by conv)
            // (eligibility again: a fusion pass may have changed the step, as
            // the global-pool fold does)
            for (Step& st : P->steps)
                if (st.kind == ST_CONV && st.u_off >= 0 && wino_eligible(st.cs)) {
                    st.wino = true;
                    st.wc = choose_wino_config(st.cs);
                    if (!(flags & NEO_PLAN_HOST_ONLY)) (void)tuned_wino_config(st.cs, &st.wc);
                }
        }
    } catch (const std::bad_alloc&) {
        rc = fail(NEO_ERR_OOM, "neo_plan_create: host allocation failed");
    } catch (const std::exception& e) {
        rc = fail(NEO_ERR_INVALID_ARG, std::string("neo_plan_create: ") + e.what());
    }
    if (rc != NEO_OK) {
        if (P->cap_stream) (void)hipStreamDestroy(P->cap_stream);
        delete P;
        return rc;
    }
    if (!(flags & NEO_PLAN_HOST_ONLY)) {
        hipError_t e = hipMalloc(&P->d_params, std::max<size_t>(P->params.size() * 4, 256));
        if (e != hipSuccess) {
            delete P;
            return e == hipErrorOutOfMemory ? fail(NEO_ERR_OOM, "neo_plan_create: parameter allocation")
                                            : hip_fail(e, "neo_plan_create: hipMalloc");
        }
        e = hipMalloc(&P->d_act, std::max<long>(P->act_bytes, 256));
        if (e != hipSuccess) {
            (void)hipFree(P->d_params);
            delete P;
            return e == hipErrorOutOfMemory ? fail(NEO_ERR_OOM, "neo_plan_create: activation allocation")
                                            : hip_fail(e, "neo_plan_create: hipMalloc");
        }
        e = hipMemcpy(P->d_params, P->params.data(), P->params.size() * 4, hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(P->d_params);
            (void)hipFree(P->d_act);
            delete P;
            return hip_fail(e, "neo_plan_create: parameter upload");
        }
        if (flags & NEO_PLAN_INT8) {
            // the packed int8 filters and their scales, from the folded filters
            e = hipMalloc(&P->d_i8, std::max<long>(P->i8_bytes, 256));
            // zero once: the halos of the inputs a producer writes directly
            // are never written again
            if (e == hipSuccess) e = hipMemset(P->d_i8, 0, std::max<long>(P->i8_bytes, 256));
            if (e == hipSuccess) e = hipMalloc(&P->d_absmax, 256);
            // (every integer conv: the steps' and the group launches' members)
            auto pack = [&](const Step& st) {
                if (e == hipSuccess && st.kind == ST_CONV && st.i8) {
                    const ConvShape s8 = int8_conv_shape(st);  // (im2col: the K(RS)C filter as 1x1)
                    e = launch_pack_filter_int8(P->d_params + st.kcrs_off, s8.K, s8.C, s8.R, s8.S,
                                                P->d_i8 + st.w8_off, P->d_params + st.ws8_off, nullptr);
                }
                if (e == hipSuccess && st.kind == ST_DENSE && st.i8)
                    e = st.d_conv  // [OUT][IN] float32 is KCRS with R = S = 1
                            ? launch_pack_filter_int8(P->d_params + st.w_off, st.dense_out, st.dense_in, 1, 1,
                                                      P->d_i8 + st.w8_off, P->d_params + st.ws8_off, nullptr)
                            : launch_pack_dense_int8(P->d_params + st.w_off, st.dense_out, st.dense_in,
                                                     P->d_i8 + st.w8_off, P->d_params + st.ws8_off, nullptr);
            };
            for (const Step& st : P->steps) {
                pack(st);
                for (const Step& m : st.members) pack(m);
            }
            if (e == hipSuccess) e = hipDeviceSynchronize();
            if (e != hipSuccess) {
                if (P->d_i8) (void)hipFree(P->d_i8);
                if (P->d_absmax) (void)hipFree(P->d_absmax);
                (void)hipFree(P->d_params);
                (void)hipFree(P->d_act);
                delete P;
                return e == hipErrorOutOfMemory ? fail(NEO_ERR_OOM, "neo_plan_create: int8 arena")
                                                : hip_fail(e, "neo_plan_create: int8 filter packing");
            }
        }
        if (flags & NEO_PLAN_TUNE) {
            const int trc = tune_plan(P);
            if (trc != NEO_OK) {
                (void)hipFree(P->d_params);
                (void)hipFree(P->d_act);
                if (P->cap_stream) (void)hipStreamDestroy(P->cap_stream);
                delete P;
                return trc;
            }
        }
        for (const Step& st : P->steps)
            if (st.kind == ST_CONV)
                P->ws_bytes = std::max(P->ws_bytes, conv_workspace_bytes(st.cs, st.wino ? st.wc : st.cc));
        if (P->ws_bytes) e = hipMalloc(&P->d_ws, P->ws_bytes);
        if (e != hipSuccess) {
            (void)hipFree(P->d_params);
            (void)hipFree(P->d_act);
            if (P->cap_stream) (void)hipStreamDestroy(P->cap_stream);
            delete P;
            return fail(NEO_ERR_OOM, "neo_plan_create: workspace");
        }
    }
    {
        std::lock_guard<std::mutex> lk(g_plans_mu);
        g_plans.insert(P);
    }
    *out = P;
    return NEO_OK;
}

int neo_plan_describe(const neo_plan* plan, char* buf, size_t len) {
    if (!live(plan)) return fail(NEO_ERR_STATE, "neo_plan_describe: not a live plan");
    const std::string s = describe(plan);
    if (buf && len) {
        const size_t n = std::min(len - 1, s.size());
        std::memcpy(buf, s.data(), n);
        buf[n] = 0;
    }
    return (int)s.size();
}

int neo_plan_output_shape(const neo_plan* plan, int* dims) {
    if (!live(plan)) return fail(NEO_ERR_STATE, "neo_plan_output_shape: not a live plan");
    if (!dims) return fail(NEO_ERR_INVALID_ARG, "neo_plan_output_shape: dims is NULL");
    for (int i = 0; i < 4; ++i) dims[i] = plan->out_dims[i];
    return NEO_OK;
}

int neo_plan_conv_params(const neo_plan* plan, int node_id, float* w_packed, float* bias) {
    if (!live(plan)) return fail(NEO_ERR_STATE, "neo_plan_conv_params: not a live plan");
    std::vector<const Step*> convs;
    for (const Step& s : plan->steps) {
        if (s.kind == ST_CONV) convs.push_back(&s);
        for (const Step& m : s.members) convs.push_back(&m);
    }
    for (const Step* sp : convs) {
        const Step& s = *sp;
        if (s.node != node_id) continue;
        if (w_packed) from_kernel_order(plan->params.data() + s.w_off, s.cs, w_packed);
        if (bias) {
            const long bn = (long)cdiv(s.cs.K, 16) * 16;
            if (s.b_off >= 0)
                std::copy(plan->params.begin() + s.b_off, plan->params.begin() + s.b_off + bn, bias);
            else
                std::fill(bias, bias + bn, 0.f);
        }
        return NEO_OK;
    }
    return fail(NEO_ERR_INVALID_ARG, "neo_plan_conv_params: node is not a conv of this plan");
}

// An integer conv step's operands and outputs (its input's int8 copy, the
// packed filter and scales, the float32 output and/or the copy it writes).
static I8Member i8_member(const neo_plan* P, const Step& s, const float* x_nchw, float* y_out) {
    const I8Copy& qc = P->i8_copies[s.qc];
    const I8Copy* qo = (s.q_out >= 0 && !P->i8_f32_out) ? &P->i8_copies[s.q_out] : nullptr;
    I8Member m;
    m.s = int8_conv_shape(s);
    m.x = P->d_i8 + qc.xq_off;
    m.w = P->d_i8 + s.w8_off;
    m.wscale = P->d_params + s.ws8_off;
    m.xscale = qc.xscale;
    m.bias = s.b_off >= 0 ? P->d_params + s.b_off : nullptr;
    m.res = s.res >= 0 ? val_ptr(P, s.res, x_nchw, y_out) : nullptr;
    m.y = (!qo || s.f32_needed) ? val_ptr(P, s.out, x_nchw, y_out) : nullptr;
    m.yq = qo ? P->d_i8 + qo->xq_off : nullptr;
    m.yscale = qo ? qo->xscale : 1.f;
    m.qph = qo ? qo->ph : 0;
    m.qpw = qo ? qo->pw : 0;
    m.xph = qc.ph;
    m.xpw = qc.pw;
    m.q_off = qo ? s.q_off8 : -1;
    m.q_tot = qo ? s.q_tot8 : -1;
    m.ydivide = qo && qo->divide;
    return m;
}

// The quantization pass of an integer conv step's input copy, if it runs it.
static hipError_t i8_quant_pass(const neo_plan* P, const Step& s, const float* x_nchw, float* y_out,
                                hipStream_t st) {
    if (!s.quant_here) return hipSuccess;
    const Val& in = P->vals[s.in];
    const I8Copy& qc = P->i8_copies[s.qc];
    if (qc.im2col)
        return launch_im2col_int8(val_ptr(P, qc.src >= 0 ? qc.src : s.in, x_nchw, y_out), qc.src >= 0, qc.ics,
                                  qc.xscale, P->d_i8 + qc.xq_off, st);
    if (qc.rows)
        return launch_quantize_rows_int8(val_ptr(P, s.in, x_nchw, y_out), in.N, in.C * in.H * in.W, qc.xscale,
                                         P->d_i8 + qc.xq_off, st);
    return launch_quantize_int8(val_ptr(P, s.in, x_nchw, y_out), in.N, in.C, in.H, in.W, qc.ph, qc.pw,
                                qc.xscale, P->d_i8 + qc.xq_off, st);
}

static int enqueue_step(neo_plan* P, const Step& s, const float* x_nchw, float* y_out,
                        hipStream_t st) {
    {
        hipError_t e = hipSuccess;
        const float* prm = P->d_params;
        switch (s.kind) {
            case ST_TRANSFORM: {
                const Val& in = P->vals[s.in];
                const Val& out = P->vals[s.out];
                float* dst = val_ptr(P, s.out, x_nchw, y_out);
                if (s.q_out >= 0 && !P->i8_f32_out) {
                    // NEO_PLAN_INT8: NCHW16c -> NCHW also as the dense layer's int8 rows
                    const I8Copy& qo = P->i8_copies[s.q_out];
                    e = launch_blk_to_rows_int8(val_ptr(P, s.in, x_nchw, y_out), in.N, in.C, in.H, in.W,
                                                s.f32_needed ? dst : nullptr, P->d_i8 + qo.xq_off, qo.xscale, st);
                    break;
                }
                e = launch_layout_transform(val_ptr(P, s.in, x_nchw, y_out), in.layout, dst,
                                            out.layout, in.N, in.C, in.H, in.W, out.c_off,
                                            out.c_tot, st);
                break;
            }
            case ST_CONV:
                if (s.i8) {
                    // the input's int8 copy (quantized here by the first
                    // reader, unless its producer wrote it), the integer conv,
                    // its float32 output and/or the int8 copy it writes
                    e = i8_quant_pass(P, s, x_nchw, y_out, st);
                    if (e == hipSuccess) e = launch_conv_int8_m(i8_member(P, s, x_nchw, y_out), s.c8, st);
                    break;
                }
                if (s.wino) {
                    e = launch_wino(s.cs, s.wc, val_ptr(P, s.in, x_nchw, y_out), prm + s.u_off,
                                    s.b_off >= 0 ? prm + s.b_off : nullptr,
                                    s.res >= 0 ? val_ptr(P, s.res, x_nchw, y_out) : nullptr,
                                    val_ptr(P, s.out, x_nchw, y_out), P->d_ws, st);
                    break;
                }
                e = launch_conv2d(s.cs, s.cc, val_ptr(P, s.in, x_nchw, y_out), prm + s.w_off, true,
                                  s.b_off >= 0 ? prm + s.b_off : nullptr,
                                  s.res >= 0 ? val_ptr(P, s.res, x_nchw, y_out) : nullptr,
                                  val_ptr(P, s.out, x_nchw, y_out), P->d_ws, st);
                break;
            case ST_CONV_GROUP: {
                const int n = (int)s.members.size();
                GroupPool gp;
                const bool has_pool = group_pool(P, s, x_nchw, y_out, &gp);
                if (s.i8) {
                    // the members' quantization passes, then one launch
                    I8Member mem[kMaxGroupConvs];
                    for (int m = 0; m < n && e == hipSuccess; ++m) {
                        e = i8_quant_pass(P, s.members[m], x_nchw, y_out, st);
                        mem[m] = i8_member(P, s.members[m], x_nchw, y_out);
                    }
                    if (e == hipSuccess) e = launch_conv_int8_group(mem, n, s.c8, has_pool ? &gp : nullptr, st);
                    break;
                }
                ConvShape shp[kMaxGroupConvs];
                const float *xs[kMaxGroupConvs], *ws[kMaxGroupConvs], *bs[kMaxGroupConvs], *rs[kMaxGroupConvs];
                float* ys[kMaxGroupConvs];
                for (int m = 0; m < n; ++m) {
                    const Step& ms = s.members[m];
                    shp[m] = ms.cs;
                    xs[m] = val_ptr(P, ms.in, x_nchw, y_out);
                    ws[m] = prm + ms.w_off;
                    bs[m] = ms.b_off >= 0 ? prm + ms.b_off : nullptr;
                    rs[m] = ms.res >= 0 ? val_ptr(P, ms.res, x_nchw, y_out) : nullptr;
                    ys[m] = val_ptr(P, ms.out, x_nchw, y_out);
                }
                e = launch_conv_group(shp, n, s.cc, xs, ws, bs, rs, ys, has_pool ? &gp : nullptr, st);
                break;
            }
            case ST_CONV_PAIR: {
                const Step &a = s.members[0], &b = s.members[1];
                e = launch_conv_pair(a.cs, b.cs, val_ptr(P, a.in, x_nchw, y_out), prm + a.w_off,
                                     a.b_off >= 0 ? prm + a.b_off : nullptr,
                                     a.res >= 0 ? val_ptr(P, a.res, x_nchw, y_out) : nullptr,
                                     val_ptr(P, a.out, x_nchw, y_out), prm + b.w_off,
                                     b.b_off >= 0 ? prm + b.b_off : nullptr,
                                     val_ptr(P, b.out, x_nchw, y_out), st);
                break;
            }
            case ST_CONV_CHAIN: {
                const int n = (int)s.members.size();
                ConvShape shp[3];
                for (int m = 0; m < n; ++m) shp[m] = s.members[m].cs;
                const Step &c = s.members[0], &a = s.members[1], &b = s.members[n - 1];
                e = launch_conv_chain(shp, n, val_ptr(P, c.in, x_nchw, y_out), prm + c.w_off,
                                      c.b_off >= 0 ? prm + c.b_off : nullptr, prm + a.w_off,
                                      a.b_off >= 0 ? prm + a.b_off : nullptr,
                                      a.res >= 0 ? val_ptr(P, a.res, x_nchw, y_out) : nullptr,
                                      val_ptr(P, a.out, x_nchw, y_out), n == 3 ? prm + b.w_off : nullptr,
                                      n == 3 && b.b_off >= 0 ? prm + b.b_off : nullptr,
                                      n == 3 ? val_ptr(P, b.out, x_nchw, y_out) : nullptr, st);
                break;
            }
            case ST_CONV_POOL: {
                const Step& c = s.members[0];
                e = launch_conv_pool(c.cs, s.pools[0].ps, s.cpc, val_ptr(P, c.in, x_nchw, y_out),
                                     prm + c.w_off, c.b_off >= 0 ? prm + c.b_off : nullptr,
                                     val_ptr(P, s.out, x_nchw, y_out), st);
                break;
            }
            case ST_MAXPOOL:
            case ST_AVGPOOL:
                if (s.q_out >= 0 && !P->i8_f32_out) {
                    // NEO_PLAN_INT8: the pool writes the int8 copy its conv readers share
                    const I8Copy& qo = P->i8_copies[s.q_out];
                    PoolQ q;
                    q.yq = P->d_i8 + qo.xq_off;
                    q.scale = qo.xscale;
                    q.qph = qo.ph;
                    q.qpw = qo.pw;
                    q.q_off = s.q_off8 >= 0 ? s.q_off8 : 0;
                    q.q_tot = s.q_tot8 > 0 ? s.q_tot8 : 0;
                    if (s.p8 >= 0)  // from its conv's int8 output
                        e = launch_maxpool_i8(s.ps, P->d_i8 + P->i8_copies[s.p8].xq_off, q, st);
                    else
                        e = launch_pool_q(s.ps, s.kind == ST_MAXPOOL, val_ptr(P, s.in, x_nchw, y_out),
                                          s.f32_needed ? val_ptr(P, s.out, x_nchw, y_out) : nullptr, q, st);
                } else if (s.kind == ST_MAXPOOL) {
                    e = launch_maxpool(s.ps, val_ptr(P, s.in, x_nchw, y_out), val_ptr(P, s.out, x_nchw, y_out), st);
                } else {
                    e = launch_avgpool(s.ps, val_ptr(P, s.in, x_nchw, y_out), val_ptr(P, s.out, x_nchw, y_out), st);
                }
                break;
            case ST_GAP: {
                const Val& in = P->vals[s.in];
                if (s.q_out >= 0 && !P->i8_f32_out) {
                    // NEO_PLAN_INT8: the means also as the dense layer's int8 rows
                    const I8Copy& qo = P->i8_copies[s.q_out];
                    e = launch_gap_q(val_ptr(P, s.in, x_nchw, y_out), in.N, in.C, in.H, in.W,
                                     s.f32_needed ? val_ptr(P, s.out, x_nchw, y_out) : nullptr,
                                     P->d_i8 + qo.xq_off, qo.xscale, st);
                    break;
                }
                e = launch_gap(val_ptr(P, s.in, x_nchw, y_out), in.layout, in.N, in.C, in.H, in.W,
                               val_ptr(P, s.out, x_nchw, y_out), st);
                break;
            }
            case ST_DENSE: {
                const Val& in = P->vals[s.in];
                if (s.i8) {
                    // the input's int8 rows (quantized here by the first
                    // reader, unless the producing dense layer wrote them),
                    // the integer dense layer, its float32 output and/or the
                    // next dense layer's int8 rows
                    const I8Copy& qc = P->i8_copies[s.qc];
                    const I8Copy* qo = (s.q_out >= 0 && !P->i8_f32_out) ? &P->i8_copies[s.q_out] : nullptr;
                    e = i8_quant_pass(P, s, x_nchw, y_out, st);
                    if (e == hipSuccess && s.d_conv)
                        e = launch_conv_int8_m(i8_member(P, s, x_nchw, y_out), s.c8, st);
                    else if (e == hipSuccess)
                        e = launch_dense_int8(P->d_i8 + qc.xq_off, P->d_i8 + s.w8_off, prm + s.ws8_off, qc.xscale,
                                              s.b_off >= 0 ? prm + s.b_off : nullptr, in.N, s.dense_in,
                                              s.dense_out, s.act,
                                              (!qo || s.f32_needed) ? val_ptr(P, s.out, x_nchw, y_out) : nullptr,
                                              qo ? P->d_i8 + qo->xq_off : nullptr, qo ? qo->xscale : 1.f, st);
                    break;
                }
                if (s.gap_parts)
                    e = launch_dense_parts(val_ptr(P, s.in, x_nchw, y_out), s.gap_parts, s.gap_stride,
                                           s.gap_scale, s.dense_in, prm + s.w_off, s.dense_out,
                                           s.b_off >= 0 ? prm + s.b_off : nullptr, s.act,
                                           val_ptr(P, s.out, x_nchw, y_out), st);
                else
                    e = launch_dense(val_ptr(P, s.in, x_nchw, y_out), in.N, s.dense_in, prm + s.w_off,
                                     s.dense_out, s.b_off >= 0 ? prm + s.b_off : nullptr, s.act,
                                     val_ptr(P, s.out, x_nchw, y_out), st);
                break;
            }
            case ST_COPY: {
                const Val& o = P->vals[s.in];
                const long bytes = (long)o.N * o.C * o.H * o.W * 4;
                e = hipMemcpyAsync(y_out, val_ptr(P, s.in, x_nchw, y_out), bytes,
                                   hipMemcpyDeviceToDevice, st);
                break;
            }
        }
        if (e != hipSuccess) return hip_fail(e, "neo_run_graph: launch");
    }
    return NEO_OK;
}

static int enqueue_steps(neo_plan* P, const float* x_nchw, float* y_out, hipStream_t st) {
    for (const Step& s : P->steps) {
        const int rc = enqueue_step(P, s, x_nchw, y_out, st);
        if (rc != NEO_OK) return rc;
    }
    return NEO_OK;
}

// Local search for every conv step (NEO_PLAN_TUNE), with the plan's own
// buffers, on its private stream; then size the split workspace for the
// chosen configurations.
static int tune_plan(neo_plan* P) {
    hipError_t e;
    if (!P->cap_stream) {
        e = hipStreamCreateWithFlags(&P->cap_stream, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "neo_plan_create: tuning stream");
    }
    // stand-in input / output of the network's shapes (contents do not matter)
    const Val& in = P->vals[P->input_val];
    const Val& out = P->vals[P->out_val];
    float *xin = nullptr, *yout = nullptr;
    e = hipMalloc(&xin, std::max<size_t>((size_t)in.N * in.C * in.H * in.W * 4, 256));
    if (e == hipSuccess) e = hipMalloc(&yout, std::max<size_t>((size_t)out.N * out.C * out.H * out.W * 4, 256));
    if (e == hipSuccess) e = hipMemset(xin, 0, (size_t)in.N * in.C * in.H * in.W * 4);
    int rc = e == hipSuccess ? NEO_OK : fail(NEO_ERR_OOM, "neo_plan_create: tuning buffers");
    // a pair stays only where it beats its two convs' own best launches;
    // appends what runs (the pair, or the two convs) and its time
    auto tune_pair = [&](const Step& s, std::vector<Step>& emit, float* us_out) -> int {
        const float* prm = P->d_params;
        Step a = s.members[0], b = s.members[1];
        const float* ba = a.b_off >= 0 ? prm + a.b_off : nullptr;
        const float* bb = b.b_off >= 0 ? prm + b.b_off : nullptr;
        const float* res = a.res >= 0 ? val_ptr(P, a.res, xin, yout) : nullptr;
        float pair_us = 0.f, a_us = 0.f, b_us = 0.f;
        int r = tune_conv_pair(a.cs, b.cs, val_ptr(P, a.in, xin, yout), prm + a.w_off, ba, res,
                               val_ptr(P, a.out, xin, yout), prm + b.w_off, bb,
                               val_ptr(P, b.out, xin, yout), P->cap_stream, &pair_us);
        if (r == NEO_OK)
            r = tune_conv(a.cs, true, val_ptr(P, a.in, xin, yout), prm + a.w_off, ba, res,
                          val_ptr(P, a.out, xin, yout), P->cap_stream, &a.cc, &a_us);
        if (r == NEO_OK)
            r = tune_conv(b.cs, true, val_ptr(P, b.in, xin, yout), prm + b.w_off, bb, nullptr,
                          val_ptr(P, b.out, xin, yout), P->cap_stream, &b.cc, &b_us);
        if (r != NEO_OK) return r;
        a.tuned = b.tuned = true;
        if (pair_us < a_us + b_us) {
            Step keep = s;
            keep.members = {a, b};
            keep.tuned = true;
            emit.push_back(keep);
            *us_out = pair_us;
        } else {
            emit.push_back(a);
            emit.push_back(b);
            *us_out = a_us + b_us;
        }
        return NEO_OK;
    };
    std::vector<Step> next;
    for (Step& s : P->steps) {
        if (rc != NEO_OK) break;
        if (s.kind == ST_CONV_GROUP && s.i8 && !s.tuned) {
            // integer convs: the group (with its pool), the group with the
            // pool alone, or every conv alone (each in its own output mode)
            const int n = (int)s.members.size();
            I8Member mem[kMaxGroupConvs];
            for (int m = 0; m < n; ++m) mem[m] = i8_member(P, s.members[m], xin, yout);
            GroupPool gp;
            const bool has_pool = group_pool(P, s, xin, yout, &gp);
            float fused_us = 0.f, split_us = 0.f, alone_us = 0.f, pool_us = 0.f;
            ConvConfig fused_cc = s.c8, split_cc = s.c8;
            rc = tune_int8_group(mem, n, has_pool ? &gp : nullptr, P->cap_stream, &fused_cc, &fused_us);
            if (rc == NEO_OK && has_pool) rc = tune_pool(gp, P->cap_stream, &pool_us);
            if (rc == NEO_OK && has_pool && n > 1)
                rc = tune_int8_group(mem, n, nullptr, P->cap_stream, &split_cc, &split_us);
            ConvConfig own[kMaxGroupConvs];
            for (int m = 0; m < n && rc == NEO_OK; ++m) {
                float us = 0.f;
                const I8Member& q = mem[m];
                rc = tune_int8(q, P->cap_stream, &own[m], &us);
                alone_us += us;
            }
            if (rc != NEO_OK) break;
            alone_us += pool_us;
            split_us += pool_us;
            const bool split_ok = has_pool && n > 1;
            Step keep = s;
            keep.tuned = true;
            if (fused_us < alone_us && (!split_ok || fused_us <= split_us)) {
                keep.c8 = fused_cc;
            } else if (split_ok && split_us < alone_us) {
                next.push_back(s.pools[0]);
                keep.pools.clear();
                keep.c8 = split_cc;
            } else {
                if (has_pool) next.push_back(s.pools[0]);
                for (int m = 0; m < n; ++m) {
                    Step ms = s.members[m];
                    ms.c8 = own[m];
                    ms.tuned = true;
                    next.push_back(ms);
                }
                continue;
            }
            for (Step& ms : keep.members) {
                ms.c8 = keep.c8;
                ms.tuned = true;
            }
            next.push_back(keep);
            continue;
        }
        if (s.kind == ST_CONV_GROUP && !s.tuned) {
            ConvShape shp[kMaxGroupConvs];
            const float *xs[kMaxGroupConvs], *ws[kMaxGroupConvs], *bs[kMaxGroupConvs], *rs[kMaxGroupConvs];
            float* ys[kMaxGroupConvs];
            const int n = (int)s.members.size();
            const float* prm = P->d_params;
            for (int m = 0; m < n; ++m) {
                const Step& ms = s.members[m];
                shp[m] = ms.cs;
                xs[m] = val_ptr(P, ms.in, xin, yout);
                ws[m] = prm + ms.w_off;
                bs[m] = ms.b_off >= 0 ? prm + ms.b_off : nullptr;
                rs[m] = ms.res >= 0 ? val_ptr(P, ms.res, xin, yout) : nullptr;
                ys[m] = val_ptr(P, ms.out, xin, yout);
            }
            GroupPool gp;
            const bool has_pool = group_pool(P, s, xin, yout, &gp);
            // candidates, each a launch list for this step's work:
            //   fused:  the convs and the pool in one launch
            //   split:  the convs in one launch, the pool alone (n > 1)
            //   alone:  every conv and the pool in launches of their own
            float fused_us = 0.f, split_us = 0.f, alone_us = 0.f, pool_us = 0.f;
            ConvConfig fused_cc = s.cc, split_cc = s.cc;
            rc = tune_conv_group(shp, n, xs, ws, bs, rs, ys, has_pool ? &gp : nullptr, P->cap_stream,
                                 &fused_cc, &fused_us);
            if (rc == NEO_OK && has_pool) rc = tune_pool(gp, P->cap_stream, &pool_us);
            if (rc == NEO_OK && has_pool && n > 1)
                rc = tune_conv_group(shp, n, xs, ws, bs, rs, ys, nullptr, P->cap_stream, &split_cc,
                                     &split_us);
            ConvConfig own[kMaxGroupConvs];
            for (int m = 0; m < n && rc == NEO_OK; ++m) {
                float us = 0.f;
                rc = tune_conv(shp[m], true, xs[m], ws[m], bs[m], rs[m], ys[m], P->cap_stream, &own[m], &us);
                alone_us += us;
            }
            if (rc != NEO_OK) break;
            alone_us += pool_us;
            split_us += pool_us;
            const bool split_ok = has_pool && n > 1;
            Step keep = s;
            keep.tuned = true;
            if (fused_us < alone_us && (!split_ok || fused_us <= split_us)) {
                keep.cc = fused_cc;
            } else if (split_ok && split_us < alone_us) {
                next.push_back(s.pools[0]);
                keep.pools.clear();
                keep.cc = split_cc;
            } else {
                if (has_pool) next.push_back(s.pools[0]);
                for (int m = 0; m < n; ++m) {
                    Step ms = s.members[m];
                    ms.cc = own[m];
                    ms.tuned = true;
                    next.push_back(ms);
                }
                continue;
            }
            for (Step& m : keep.members) {
                m.cc = keep.cc;
                m.tuned = true;
            }
            next.push_back(keep);
            continue;
        }
        if (s.kind == ST_CONV_PAIR && !s.tuned) {
            float us = 0.f;
            rc = tune_pair(s, next, &us);
            continue;
        }
        if (s.kind == ST_CONV_CHAIN && !s.tuned) {
            // the chain stays only where it beats the 3x3's own best launch
            // plus the best of the rest (the pair, or its convs alone)
            const float* prm = P->d_params;
            const int n = (int)s.members.size();
            ConvShape shp[3];
            for (int m = 0; m < n; ++m) shp[m] = s.members[m].cs;
            Step c = s.members[0];
            const Step &a = s.members[1], &b = s.members[n - 1];
            const float* ba = a.b_off >= 0 ? prm + a.b_off : nullptr;
            const float* res = a.res >= 0 ? val_ptr(P, a.res, xin, yout) : nullptr;
            float chain_us = 0.f, c_us = 0.f, rest_us = 0.f;
            rc = tune_conv_chain(shp, n, val_ptr(P, c.in, xin, yout), prm + c.w_off,
                                 c.b_off >= 0 ? prm + c.b_off : nullptr, prm + a.w_off, ba, res,
                                 val_ptr(P, a.out, xin, yout), n == 3 ? prm + b.w_off : nullptr,
                                 n == 3 && b.b_off >= 0 ? prm + b.b_off : nullptr,
                                 n == 3 ? val_ptr(P, b.out, xin, yout) : nullptr, P->cap_stream, &chain_us);
            if (rc == NEO_OK)
                rc = tune_conv(c.cs, true, val_ptr(P, c.in, xin, yout), prm + c.w_off,
                               c.b_off >= 0 ? prm + c.b_off : nullptr, nullptr, val_ptr(P, c.out, xin, yout),
                               P->cap_stream, &c.cc, &c_us);
            std::vector<Step> rest;
            if (rc == NEO_OK && n == 3) {
                Step pr = s;
                pr.kind = ST_CONV_PAIR;
                pr.node = a.node;
                pr.in = a.in;
                pr.out2 = b.out;
                pr.members = {a, b};
                rc = tune_pair(pr, rest, &rest_us);
            } else if (rc == NEO_OK) {
                Step e1 = a;
                rc = tune_conv(e1.cs, true, val_ptr(P, e1.in, xin, yout), prm + e1.w_off, ba, res,
                               val_ptr(P, e1.out, xin, yout), P->cap_stream, &e1.cc, &rest_us);
                e1.tuned = true;
                rest.push_back(e1);
            }
            if (rc != NEO_OK) break;
            c.tuned = true;
            if (chain_us < c_us + rest_us) {
                Step keep = s;
                keep.tuned = true;
                keep.members[0] = c;
                for (size_t m = 1; m < keep.members.size(); ++m) keep.members[m].tuned = true;
                next.push_back(keep);
            } else {
                next.push_back(c);
                next.insert(next.end(), rest.begin(), rest.end());
            }
            continue;
        }
        if (s.kind == ST_CONV_POOL && !s.tuned) {
            // the fused launch stays only where it beats the conv's and the
            // pool's own best launches
            const float* prm = P->d_params;
            Step c = s.members[0];
            const Step& pl = s.pools[0];
            const float* bias = c.b_off >= 0 ? prm + c.b_off : nullptr;
            float fused_us = 0.f, conv_us = 0.f, pool_us = 0.f;
            ConvPoolConfig cpc = s.cpc;
            rc = tune_conv_pool(c.cs, pl.ps, val_ptr(P, c.in, xin, yout), prm + c.w_off, bias,
                                val_ptr(P, s.out, xin, yout), P->cap_stream, &cpc, &fused_us);
            if (rc == NEO_OK)
                rc = tune_conv(c.cs, true, val_ptr(P, c.in, xin, yout), prm + c.w_off, bias, nullptr,
                               val_ptr(P, c.out, xin, yout), P->cap_stream, &c.cc, &conv_us);
            if (rc == NEO_OK) {
                GroupPool gp{pl.ps, true, val_ptr(P, pl.in, xin, yout), val_ptr(P, pl.out, xin, yout)};
                rc = tune_pool(gp, P->cap_stream, &pool_us);
            }
            if (rc != NEO_OK) break;
            c.tuned = true;
            if (fused_us < conv_us + pool_us) {
                Step keep = s;
                keep.cpc = cpc;
                keep.tuned = true;
                keep.members[0] = c;
                next.push_back(keep);
            } else {
                next.push_back(c);
                next.push_back(pl);
            }
            continue;
        }
        if ((s.kind == ST_CONV || (s.kind == ST_DENSE && s.d_conv)) && s.i8) {
            // an integer conv (or a dense layer run as one): its configurations
            // timed with its own output mode
            rc = tune_int8(i8_member(P, s, xin, yout), P->cap_stream, &s.c8, nullptr);
            s.tuned = rc == NEO_OK;
            next.push_back(s);
            continue;
        }
        // (a conv the Winograd kernel could run is compared even when its
        // direct configuration came from the results database)
        if (s.kind == ST_CONV && (!s.tuned || s.u_off >= 0)) {
            const float* prm = P->d_params;
            // a conv with the global pool folded in is timed as a plain conv
            // (its launch then runs the configuration without a split)
            ConvShape ts = s.cs;
            ts.gap = 0;
            float direct_us = 0.f;
            rc = tune_conv(ts, true, val_ptr(P, s.in, xin, yout), prm + s.w_off,
                           s.b_off >= 0 ? prm + s.b_off : nullptr,
                           s.res >= 0 ? val_ptr(P, s.res, xin, yout) : nullptr,
                           val_ptr(P, s.out, xin, yout), P->cap_stream, &s.cc, &direct_us);
            if (s.cs.gap && s.cc.fp == 0) s.cc = choose_conv_config(s.cs);
            if (rc == NEO_OK && s.u_off >= 0 && wino_eligible(s.cs)) {
                // the Winograd kernel runs the step only where it measures faster
                float wino_us = 0.f;
                rc = tune_wino(s.cs, val_ptr(P, s.in, xin, yout), prm + s.u_off,
                               s.b_off >= 0 ? prm + s.b_off : nullptr,
                               s.res >= 0 ? val_ptr(P, s.res, xin, yout) : nullptr,
                               val_ptr(P, s.out, xin, yout), P->cap_stream, &s.wc, &wino_us);
                s.wino = rc == NEO_OK && wino_us < direct_us;
            }
            s.tuned = rc == NEO_OK;
        }
        next.push_back(s);
    }
    if (rc == NEO_OK) P->steps.swap(next);
    // groups the search split up: their convs' quantization passes again at
    // each copy's first reader
    if (rc == NEO_OK && (P->flags & NEO_PLAN_INT8)) place_int8_quant_passes(P);
    if (xin) (void)hipFree(xin);
    if (yout) (void)hipFree(yout);
    return rc;
}

static void drop_graph(neo_plan* P) {
    if (P->graph_exec) (void)hipGraphExecDestroy(P->graph_exec);
    P->graph_exec = nullptr;
    P->graph_x = nullptr;
    P->graph_y = nullptr;
}

// Capture the launch list for (x, y) on the plan's private stream.
static int capture(neo_plan* P, const float* x_nchw, float* y_out) {
    drop_graph(P);
    hipError_t e;
    if (!P->cap_stream) {
        e = hipStreamCreateWithFlags(&P->cap_stream, hipStreamNonBlocking);
        if (e != hipSuccess) return hip_fail(e, "neo_run_graph: capture stream");
    }
    e = hipStreamBeginCapture(P->cap_stream, hipStreamCaptureModeThreadLocal);
    if (e != hipSuccess) return hip_fail(e, "neo_run_graph: begin capture");
    const int rc = enqueue_steps(P, x_nchw, y_out, P->cap_stream);
    hipGraph_t g = nullptr;
    e = hipStreamEndCapture(P->cap_stream, &g);
    if (rc != NEO_OK) {
        if (g) (void)hipGraphDestroy(g);
        return rc;
    }
    if (e != hipSuccess) return hip_fail(e, "neo_run_graph: end capture");
    e = hipGraphInstantiate(&P->graph_exec, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) {
        P->graph_exec = nullptr;
        return hip_fail(e, "neo_run_graph: instantiate");
    }
    P->graph_x = x_nchw;
    P->graph_y = y_out;
    return NEO_OK;
}

int neo_run_graph(neo_plan* P, const float* x_nchw, float* y_out, neo_stream_t stream) {
    if (!live(P)) return fail(NEO_ERR_STATE, "neo_run_graph: not a live plan");
    if (P->flags & NEO_PLAN_HOST_ONLY) return fail(NEO_ERR_STATE, "neo_run_graph: host-only plan");
    if (!x_nchw || !y_out) return fail(NEO_ERR_INVALID_ARG, "neo_run_graph: NULL buffer");
    if (!aligned16(x_nchw) || !aligned16(y_out))
        return fail(NEO_ERR_ALIGN, "neo_run_graph: buffers must be 16-byte aligned");
    if ((P->flags & NEO_PLAN_INT8) && !P->i8_ready)
        return fail(NEO_ERR_STATE, "neo_run_graph: an int8 plan runs after neo_plan_calibrate_int8");
    hipStream_t st = (hipStream_t)stream;
    if (!(P->flags & NEO_PLAN_HIPGRAPH)) return enqueue_steps(P, x_nchw, y_out, st);
    if (!P->graph_exec || P->graph_x != x_nchw || P->graph_y != y_out) {
        const int rc = capture(P, x_nchw, y_out);
        if (rc != NEO_OK) return rc;
    }
    hipError_t e = hipGraphLaunch(P->graph_exec, st);
    return e == hipSuccess ? NEO_OK : hip_fail(e, "neo_run_graph: graph launch");
}

int neo_run_step(neo_plan* P, int step, const float* x_nchw, float* y_out, neo_stream_t stream) {
    if (!live(P)) return fail(NEO_ERR_STATE, "neo_run_step: not a live plan");
    if (P->flags & NEO_PLAN_HOST_ONLY) return fail(NEO_ERR_STATE, "neo_run_step: host-only plan");
    if (step < 0 || step >= (int)P->steps.size())
        return fail(NEO_ERR_INVALID_ARG, "neo_run_step: step out of range");
    if (!x_nchw || !y_out) return fail(NEO_ERR_INVALID_ARG, "neo_run_step: NULL buffer");
    if (!aligned16(x_nchw) || !aligned16(y_out))
        return fail(NEO_ERR_ALIGN, "neo_run_step: buffers must be 16-byte aligned");
    if ((P->flags & NEO_PLAN_INT8) && !P->i8_ready)
        return fail(NEO_ERR_STATE, "neo_run_step: an int8 plan runs after neo_plan_calibrate_int8");
    return enqueue_step(P, P->steps[step], x_nchw, y_out, (hipStream_t)stream);
}

int neo_plan_calibrate_int8(neo_plan* P, const float* x_nchw, float* y_out, neo_stream_t stream) {
    if (!live(P)) return fail(NEO_ERR_STATE, "neo_plan_calibrate_int8: not a live plan");
    if (!(P->flags & NEO_PLAN_INT8) || (P->flags & NEO_PLAN_HOST_ONLY))
        return fail(NEO_ERR_STATE, "neo_plan_calibrate_int8: not a device plan with NEO_PLAN_INT8");
    if (!x_nchw || !y_out) return fail(NEO_ERR_INVALID_ARG, "neo_plan_calibrate_int8: NULL buffer");
    if (!aligned16(x_nchw) || !aligned16(y_out))
        return fail(NEO_ERR_ALIGN, "neo_plan_calibrate_int8: buffers must be 16-byte aligned");
    hipStream_t st = (hipStream_t)stream;
    drop_graph(P);
    P->i8_ready = false;
    // max |x| / 127 in float32 over n floats of the device tensor x (1 for zeros)
    auto scale_of = [&](const float* x, long n, float* out) {
        unsigned bits = 0;
        hipError_t e = launch_absmax(x, n, P->d_absmax, st);
        if (e == hipSuccess) e = hipMemcpyAsync(&bits, P->d_absmax, 4, hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return hip_fail(e, "neo_plan_calibrate_int8: input maximum");
        float m;
        std::memcpy(&m, &bits, 4);
        if (!std::isfinite(m)) return fail(NEO_ERR_INVALID_ARG, "neo_plan_calibrate_int8: non-finite activation");
        *out = m > 0.f ? m / 127.0f : 1.0f;
        return (int)NEO_OK;
    };
    auto elems = [&](int v) {  // the floats of a value (blocked: with its padding lanes)
        const Val& a = P->vals[v];
        return a.layout ? (long)a.N * cdiv(a.C, a.layout) * a.layout * a.H * a.W : (long)a.N * a.C * a.H * a.W;
    };
    // an assembled copy's parts (the steps writing its slices; group members
    // with their group's configuration), and whether its scale is set
    std::vector<std::vector<Step>> parts(P->i8_copies.size());
    for (const Step& t : P->steps) {
        auto add = [&](const Step& x, const ConvConfig* c8) {
            if (x.q_out < 0 || !P->i8_copies[x.q_out].assembled) return;
            Step one = x;
            if (c8) one.c8 = *c8;
            parts[x.q_out].push_back(one);
        };
        add(t, nullptr);
        for (const Step& m : t.members) add(m, t.i8 ? &t.c8 : nullptr);
        for (const Step& pl : t.pools) add(pl, nullptr);
    }
    std::vector<char> assembled(P->i8_copies.size(), 0);
    // one step as the calibration runs it: a group's members (and its pool)
    // one by one, which computes what the group launch does
    std::function<int(const Step&)> calibrate_step = [&](const Step& s) -> int {
        if (s.kind == ST_CONV_GROUP && s.i8) {
            for (const Step& m : s.members) {
                Step one = m;
                one.c8 = s.c8;
                const int rc = calibrate_step(one);
                if (rc != NEO_OK) return rc;
            }
            for (const Step& pl : s.pools) {
                const int rc = calibrate_step(pl);
                if (rc != NEO_OK) return rc;
            }
            return NEO_OK;
        }
        int rc;
        if (s.kind == ST_CONV && s.i8 && P->i8_copies[s.qc].assembled && !assembled[s.qc]) {
            // the first reader of an assembled copy: every part has run in
            // float32; the scale of the whole concatenation, then the parts
            // again, now writing their slices
            I8Copy& q = P->i8_copies[s.qc];
            if ((rc = scale_of(val_ptr(P, q.val, x_nchw, y_out), elems(q.val), &q.xscale)) != NEO_OK) return rc;
            for (const Step& part : parts[s.qc])
                if ((rc = enqueue_step(P, part, x_nchw, y_out, st)) != NEO_OK) return rc;
            assembled[s.qc] = 1;
        }
        // a copy quantized by its own pass: the scale of the value it reads
        // (an im2col pass from the NCHW value: that value's)
        if ((s.kind == ST_CONV || s.kind == ST_DENSE) && s.i8 && s.quant_here) {
            const int src = P->i8_copies[s.qc].src >= 0 ? P->i8_copies[s.qc].src : s.in;
            if ((rc = scale_of(val_ptr(P, src, x_nchw, y_out), elems(src), &P->i8_copies[s.qc].xscale)) !=
                NEO_OK)
                return rc;
        }
        if (s.q_out >= 0 && P->i8_copies[s.q_out].assembled) {
            // a part of an assembled copy: float32 only until the copy's scale is known
            P->i8_f32_out = true;
            rc = enqueue_step(P, s, x_nchw, y_out, st);
            P->i8_f32_out = false;
            return rc;
        }
        if (s.q_out >= 0) {
            // a copy's writer (conv or pool): run it once with its float32
            // output only, take the copy's scale from that, then run it as
            // the plan does
            P->i8_f32_out = true;
            rc = enqueue_step(P, s, x_nchw, y_out, st);
            P->i8_f32_out = false;
            if (rc != NEO_OK) return rc;
            I8Copy& qo = P->i8_copies[s.q_out];
            if (qo.pool_copy >= 0) {
                // a max pool's int8 input: the pool's float32 output gives
                // the scale of both copies
                for (const Step& pl : P->steps)
                    if (pl.p8 == s.q_out) {
                        P->i8_f32_out = true;
                        rc = enqueue_step(P, pl, x_nchw, y_out, st);
                        P->i8_f32_out = false;
                        if (rc != NEO_OK) return rc;
                        if ((rc = scale_of(val_ptr(P, pl.out, x_nchw, y_out), elems(pl.out),
                                           &P->i8_copies[qo.pool_copy].xscale)) != NEO_OK)
                            return rc;
                        qo.xscale = P->i8_copies[qo.pool_copy].xscale;
                    }
            } else if ((rc = scale_of(val_ptr(P, s.out, x_nchw, y_out), elems(s.out), &qo.xscale)) != NEO_OK) {
                return rc;
            }
        }
        return enqueue_step(P, s, x_nchw, y_out, st);
    };
    for (const Step& s : P->steps) {
        const int rc = calibrate_step(s);
        if (rc != NEO_OK) return rc;
    }
    hipError_t e = hipStreamSynchronize(st);
    if (e != hipSuccess) return hip_fail(e, "neo_plan_calibrate_int8: run");
    P->i8_ready = true;
    return NEO_OK;
}

void neo_plan_destroy(neo_plan* plan) {
    {
        std::lock_guard<std::mutex> lk(g_plans_mu);
        if (!plan || !g_plans.count(plan)) return;
        g_plans.erase(plan);
    }
    if (plan->d_params || plan->d_act) {
        (void)hipDeviceSynchronize();
        drop_graph(plan);
        if (plan->cap_stream) (void)hipStreamDestroy(plan->cap_stream);
        (void)hipFree(plan->d_params);
        (void)hipFree(plan->d_act);
        if (plan->d_ws) (void)hipFree(plan->d_ws);
        if (plan->d_i8) (void)hipFree(plan->d_i8);
        if (plan->d_absmax) (void)hipFree(plan->d_absmax);
    }
    delete plan;
}

}  // extern "C"
