// Global layout search (Section 3.3.2, Algorithm 2).
//
// Every convolution chooses a scheme, the split factors (ic_bn, oc_bn) of its
// input and output layouts; each scheme has an execution time from the local
// search, and each choice implies layout transforms wherever a producer's
// layout differs from what a consumer reads.  The program visits the nodes in
// topological order and, for every combination of layouts of the values that
// are still to be read later, memorises the cheapest way to reach it: a
// convolution's scheme j costs its execution time plus the transforms from
// the layouts its inputs have (the predecessors' memorised schemes k) to the
// ones j reads, added to the predecessors' optima.  On a list-shaped network
// the state is the previous convolution's output layout and this is exactly
// the recurrence of Algorithm 2; on a graph where a value is read again later
// (a residual, a branch to concatenate), that value's layout stays in the
// state until its last reader -- the schemes the paper says must be saved for
// a future use -- which keeps the program exact.  The state also records which
// layouts a value has already been transformed to, because the plan transforms
// a value once per layout and every later reader of that layout shares it.
//
// Layout rules (the planner's, see plan.cpp): a conv reads its input in
// ic_bn and its residual in oc_bn and writes oc_bn; pooling runs in its
// input's layout (the default block if that is NCHW); a concat takes its first
// input's layout when every part is a whole number of its blocks (else the
// default block, else NCHW) and converts the other parts; flatten, dense and
// the output need NCHW.  A transform of a 1x1 map whose channel count both
// blocks divide is an alias and costs nothing, except into a concat.
#include <algorithm>
#include <cmath>
#include <map>
#include <vector>

#include "neo_internal.h"

namespace neo {

const int kSearchBlocks[NEO_SEARCH_NB] = {0, 4, 8, 16, 32, 64};

int search_block_index(int block) {
    for (int i = 0; i < NEO_SEARCH_NB; ++i)
        if (kSearchBlocks[i] == block) return i;
    return -1;
}

bool layout_alias(int C, int H, int W, int src, int dst, bool into_concat) {
    if (into_concat || H * W != 1) return false;
    return (src == 0 || C % src == 0) && (dst == 0 || C % dst == 0);
}

namespace {

constexpr int NB = NEO_SEARCH_NB;
constexpr long kMaxStates = 1L << 20;

struct Live {
    int val, nat, have;  // value (node id), its layout (block index), layouts it has (bit mask)
};
using Key = std::vector<int>;  // (val, nat, have) triples, sorted by val

struct Entry {
    double cost;
    int prev;    // index of the state in the previous layer
    int choice;  // conv: ic * NB + oc; other nodes: -1
};

Key encode(std::vector<Live>& st) {
    std::sort(st.begin(), st.end(), [](const Live& a, const Live& b) { return a.val < b.val; });
    Key k;
    k.reserve(st.size() * 3);
    for (const Live& l : st) {
        k.push_back(l.val);
        k.push_back(l.nat);
        k.push_back(l.have);
    }
    return k;
}

std::vector<Live> decode(const Key& k) {
    std::vector<Live> st(k.size() / 3);
    for (size_t i = 0; i < st.size(); ++i) st[i] = Live{k[3 * i], k[3 * i + 1], k[3 * i + 2]};
    return st;
}

}  // namespace

int layout_search_dp(const std::vector<SearchNode>& g, const std::vector<int>& order,
                     int default_block, const SearchCost& conv_cost, const SearchCost& xform_cost,
                     std::vector<int>* ic, std::vector<int>* oc, double* cost, long* max_states) {
    const int n = (int)g.size();
    const int D = search_block_index(default_block);
    if (D < 0) return fail(NEO_ERR_INVALID_ARG, "layout search: bad default block");
    std::vector<int> pos(n, 0), last(n, -1);
    for (int k = 0; k < n; ++k) pos[order[k]] = k;
    for (int v : order) {
        std::vector<int> rd = g[v].inputs;
        if (g[v].residual >= 0) rd.push_back(g[v].residual);
        for (int u : rd) last[u] = std::max(last[u], pos[v]);
    }

    std::vector<std::vector<Key>> keys(n + 1);
    std::vector<std::vector<Entry>> ents(n + 1);
    keys[0].push_back(Key{});
    ents[0].push_back(Entry{0.0, -1, -1});
    long widest = 1;
    for (int k = 0; k < n; ++k) {
        const int v = order[k];
        const SearchNode& nd = g[v];
        std::vector<int> choices;
        if (nd.op == NEO_OP_CONV) {
            for (int i = 0; i < NB; ++i)
                for (int j = 0; j < NB; ++j) {
                    const double t = conv_cost(v, i, j);
                    if (std::isfinite(t) && t >= 0) choices.push_back(i * NB + j);
                }
        } else {
            choices.push_back(-1);
        }
        std::map<Key, int> index;
        for (size_t si = 0; si < keys[k].size(); ++si) {
            const std::vector<Live> base = decode(keys[k][si]);
            const double base_cost = ents[k][si].cost;
            for (int ch : choices) {
                std::vector<Live> st = base;
                double c = base_cost;
                auto find = [&](int u) -> Live* {
                    for (Live& l : st)
                        if (l.val == u) return &l;
                    return nullptr;
                };
                // reader of value u in layout L (block index)
                auto fetch = [&](int u, int L, bool into_concat) {
                    Live* l = find(u);
                    if (!l) {  // cannot happen: u is read at or after this node
                        c = INFINITY;
                        return;
                    }
                    if (l->have & (1 << L)) return;
                    l->have |= 1 << L;
                    const SearchNode& s = g[u];
                    if (!layout_alias(s.C, s.H, s.W, kSearchBlocks[l->nat], kSearchBlocks[L], into_concat))
                        c += xform_cost(u, l->nat, L);
                };
                int lay = 0;
                switch (nd.op) {
                    case NEO_OP_INPUT:
                        lay = 0;
                        break;
                    case NEO_OP_CONV: {
                        const int i = ch / NB, j = ch % NB;
                        c += conv_cost(v, i, j);
                        fetch(nd.inputs[0], i, false);
                        if (nd.residual >= 0) fetch(nd.residual, j, false);
                        lay = j;
                        break;
                    }
                    case NEO_OP_MAXPOOL:
                    case NEO_OP_AVGPOOL:
                    case NEO_OP_GAP: {
                        const Live* l = find(nd.inputs[0]);
                        lay = (l && l->nat != 0) ? l->nat : D;
                        fetch(nd.inputs[0], lay, false);
                        break;
                    }
                    case NEO_OP_CONCAT: {
                        const Live* l = find(nd.inputs[0]);
                        const int first = l ? kSearchBlocks[l->nat] : 0;
                        auto whole = [&](int b) {
                            for (int u : nd.inputs)
                                if (g[u].C % b) return false;
                            return true;
                        };
                        if (first > 0 && whole(first))
                            lay = l->nat;
                        else if (whole(default_block))
                            lay = D;
                        else
                            lay = 0;
                        for (int u : nd.inputs) fetch(u, lay, true);
                        break;
                    }
                    default:  // flatten, dense, output
                        fetch(nd.inputs[0], 0, false);
                        lay = 0;
                        break;
                }
                if (!std::isfinite(c)) continue;
                if (last[v] > k) st.push_back(Live{v, lay, 1 << lay});
                st.erase(std::remove_if(st.begin(), st.end(), [&](const Live& l) { return last[l.val] <= k; }),
                         st.end());
                Key key = encode(st);
                auto it = index.find(key);
                if (it == index.end()) {
                    index.emplace(key, (int)keys[k + 1].size());
                    keys[k + 1].push_back(std::move(key));
                    ents[k + 1].push_back(Entry{c, (int)si, ch});
                } else if (c < ents[k + 1][it->second].cost) {
                    ents[k + 1][it->second] = Entry{c, (int)si, ch};
                }
            }
        }
        if (keys[k + 1].empty())
            return fail(NEO_ERR_SHAPE, "layout search: no feasible scheme at node " + std::to_string(v));
        widest = std::max(widest, (long)keys[k + 1].size());
        if (widest > kMaxStates)
            return fail(NEO_ERR_UNSUPPORTED, "layout search: more than 2^20 states (the dynamic "
                                             "program is intractable for this graph)");
    }
    int best = 0;
    for (size_t i = 1; i < ents[n].size(); ++i)
        if (ents[n][i].cost < ents[n][best].cost) best = (int)i;
    ic->assign(n, 0);
    oc->assign(n, 0);
    if (cost) *cost = ents[n][best].cost;
    if (max_states) *max_states = widest;
    int si = best;
    for (int k = n; k > 0; --k) {
        const Entry& e = ents[k][si];
        if (e.choice >= 0) {
            (*ic)[order[k - 1]] = kSearchBlocks[e.choice / NB];
            (*oc)[order[k - 1]] = kSearchBlocks[e.choice % NB];
        }
        si = e.prev;
    }
    return NEO_OK;
}

}  // namespace neo
