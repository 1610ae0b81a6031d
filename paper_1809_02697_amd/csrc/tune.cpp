// Local search over convolution launch configurations, and its results
// database (Section 3.3.1).  The paper times every candidate schedule of a
// CONV workload on the target CPU, keeps the fastest, and stores the result
// per (workload, CPU type) so that a workload is searched once.  Here a
// schedule is a launch configuration of the blocked MFMA kernel (register
// tile, waves per workgroup, reduction split), a workload is the convolution
// shape with its input and output blocks (ic_bn, oc_bn), and the "CPU type" is
// the GPU architecture name.
#include <algorithm>
#include <cstdio>
#include <cstring>
#include <fstream>
#include <map>
#include <mutex>
#include <sstream>
#include <string>
#include <tuple>
#include <vector>

#include "neo_internal.h"

namespace neo {
namespace {

struct Key {
    std::string arch;
    int N, C, H, W, K, R, S, sh, sw, ph, pw, wmfma, xb, yb;
    auto tie() const { return std::tie(arch, N, C, H, W, K, R, S, sh, sw, ph, pw, wmfma, xb, yb); }
    bool operator<(const Key& o) const { return tie() < o.tie(); }
};

struct Entry {
    ConvConfig cfg;
    float us;
};

std::mutex g_mu;
std::map<Key, Entry> g_db;

std::string device_arch() {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return "unknown";
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return "unknown";
    std::string a = prop.gcnArchName;
    const size_t colon = a.find(':');
    return colon == std::string::npos ? a : a.substr(0, colon);
}

// The input and output blocks of a stored workload are ones the kernel takes.
bool key_blocks_valid(const Key& k) {
    ConvShape s{};
    s.C = k.C;
    s.xb = k.xb;
    s.yb = k.yb;
    return conv_blocks_valid(s);
}

Key key_of(const ConvShape& s, bool wmfma, const std::string& arch) {
    return Key{arch, s.N, s.C, s.H, s.W, s.K, s.R, s.S, s.sh, s.sw, s.ph, s.pw, wmfma ? 1 : 0,
               s.xb, s.yb};
}

// Candidate schedules: every register tile and waves-per-workgroup the kernel
// instantiates, and reduction splits that leave every wave at least one step
// and keep the partials workspace below 64 MB.
std::vector<ConvConfig> candidates(const ConvShape& s) {
    std::vector<ConvConfig> out;
    const int KB = cdiv(s.K, 16), MP = cdiv(s.N * s.OH * s.OW, 16);
    for (int fk : {1, 2, 4})
        for (int fp : {1, 2, 4})
            for (int wv : {1, 2, 4, 8, 16})
                for (int sp : {1, 2, 4, 8}) {
                    const ConvConfig c{fk, fp, sp, wv};
                    if (!conv_config_valid(c)) continue;
                    if (fk > 1 && fk > KB) continue;
                    if (fp > 1 && fp > MP) continue;
                    if (conv_steps(s, c) / sp < wv) continue;
                    if (sp > 1 && conv_workspace_bytes(s, c) > (64u << 20)) continue;
                    out.push_back(c);
                }
    return out;
}

// The streaming pointwise kernel's configurations for a shape it takes.
std::vector<ConvConfig> stream_candidates(const ConvShape& s) {
    std::vector<ConvConfig> out;
    for (int fk : {1, 2, 4})
        for (int wv : {1, 2, 4, 8}) {
            const ConvConfig c{fk, 0, 1, wv};
            if (conv_stream_config_valid(s, c)) out.push_back(c);
        }
    return out;
}

}  // namespace

bool tuned_config(const ConvShape& s, bool wmfma, ConvConfig* out) {
    const std::string arch = device_arch();
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_db.find(key_of(s, wmfma, arch));
    if (it == g_db.end()) return false;
    // a stored streaming configuration the shape cannot take is ignored
    if (it->second.cfg.fp == 0 && !conv_stream_config_valid(s, it->second.cfg)) return false;
    *out = it->second.cfg;
    return true;
}

namespace {

// one launch of several convs (and a pooling step): architecture and the
// members' shapes -> config; a pooling step alone: architecture and shape -> time
using GroupKey = std::pair<std::string, std::vector<int>>;
std::map<GroupKey, Entry> g_group_db;
std::map<GroupKey, float> g_pool_db;
std::map<GroupKey, float> g_pair_db;  // two pointwise convs in one launch -> time
std::map<GroupKey, float> g_chain_db;  // a 3x3-led chain of 2 or 3 convs in one launch -> time
struct PoolEntry {
    ConvPoolConfig cfg;
    float us;
};
std::map<GroupKey, PoolEntry> g_convpool_db;  // a stem conv and its max pool in one launch
std::map<GroupKey, Entry> g_wino_db;          // a 3x3 conv by Winograd F(2x2, 3x3)
constexpr int kWinoInts = 7;                  // N C H W K ph pw
std::map<GroupKey, Entry> g_i8_db;            // an integer conv, by output mode
constexpr int kI8Ints = 12;                   // N C H W K R S sh sw ph pw out
std::map<GroupKey, Entry> g_i8group_db;       // integer convs (and a pool) in one launch
constexpr int kConvPoolInts = 13 + 12;        // conv N C H W K R S sh sw ph pw xb act, pool ints
constexpr int kPairInts = 23;         // both convs' N C H W K R S sh sw ph pw, residual
constexpr int kGroupShapeInts = 11;  // N C H W K R S sh sw ph pw per member
constexpr int kPoolShapeInts = 12;   // max N C H W R S sh sw ph pw xb

std::vector<int> pool_ints(const GroupPool& p) {
    const PoolShape& s = p.s;
    return {p.max ? 1 : 0, s.N, s.C, s.H, s.W, s.R, s.S, s.sh, s.sw, s.ph, s.pw, s.xb};
}

}  // namespace

// Time every candidate with the caller's buffers on `st`.  Keeps the fastest
// in the database and returns it with its time per launch (us_out may be
// null).
int tune_conv(const ConvShape& s, bool wmfma, const float* x, const float* w, const float* bias,
              const float* res, float* y, hipStream_t st, ConvConfig* best_out, float* us_out) {
    const std::string arch = device_arch();
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_db.find(key_of(s, wmfma, arch));
        if (it != g_db.end()) {
            *best_out = it->second.cfg;
            if (us_out) *us_out = it->second.us;
            return NEO_OK;
        }
    }
    std::vector<ConvConfig> cands = candidates(s);
    if (wmfma)
        for (const ConvConfig& c : stream_candidates(s)) cands.push_back(c);
    size_t ws_bytes = 0;
    for (const ConvConfig& c : cands) ws_bytes = std::max(ws_bytes, conv_workspace_bytes(s, c));
    float* ws = nullptr;
    hipError_t e = hipSuccess;
    if (ws_bytes) e = hipMalloc(&ws, ws_bytes);
    if (e != hipSuccess) return fail(NEO_ERR_OOM, "tuning workspace allocation");
    ConvConfig best = choose_conv_config(s);
    float best_us = 1e30f;
    {
        Events ev;
        for (const ConvConfig& c : cands) {
            float us = 0.f;
            e = time_launch([&] { return launch_conv2d(s, c, x, w, wmfma, bias, res, y, ws, st); }, st,
                            ev.e0, ev.e1, &us);
            if (e != hipSuccess) break;
            if (us < best_us) {
                best_us = us;
                best = c;
            }
        }
        (void)hipStreamSynchronize(st);
    }
    if (ws) (void)hipFree(ws);
    if (e != hipSuccess) return hip_fail(e, "tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_db[key_of(s, wmfma, arch)] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

namespace {
GroupKey wino_key(const ConvShape& s) { return {device_arch(), {s.N, s.C, s.H, s.W, s.K, s.ph, s.pw}}; }
}  // namespace

bool tuned_wino_config(const ConvShape& s, ConvConfig* out) {
    const GroupKey key = wino_key(s);
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_wino_db.find(key);
    if (it == g_wino_db.end() || !wino_config_valid(s, it->second.cfg)) return false;
    *out = it->second.cfg;
    return true;
}

// Every valid Winograd configuration with a partials workspace below 64 MB,
// timed with the caller's buffers; keeps the fastest with its time.
int tune_wino(const ConvShape& s, const float* x, const float* u, const float* bias,
              const float* res, float* y, hipStream_t st, ConvConfig* best_out, float* us_out) {
    const GroupKey key = wino_key(s);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_wino_db.find(key);
        if (it != g_wino_db.end() && wino_config_valid(s, it->second.cfg)) {
            *best_out = it->second.cfg;
            if (us_out) *us_out = it->second.us;
            return NEO_OK;
        }
    }
    std::vector<ConvConfig> cands;
    for (int fk : {1, 2})
        for (int fp : {1, 2})
            for (int wv : {1, 2, 4, 8})
                for (int sp : {1, 2, 4, 8}) {
                    const ConvConfig c{fk, fp, sp, wv};
                    if (wino_config_valid(s, c) && conv_workspace_bytes(s, c) <= (64u << 20))
                        cands.push_back(c);
                }
    size_t ws_bytes = 0;
    for (const ConvConfig& c : cands) ws_bytes = std::max(ws_bytes, conv_workspace_bytes(s, c));
    float* ws = nullptr;
    hipError_t e = hipSuccess;
    if (ws_bytes) e = hipMalloc(&ws, ws_bytes);
    if (e != hipSuccess) return fail(NEO_ERR_OOM, "Winograd tuning workspace allocation");
    ConvConfig best = choose_wino_config(s);
    float best_us = 1e30f;
    {
        Events ev;
        for (const ConvConfig& c : cands) {
            float us = 0.f;
            e = time_launch([&] { return launch_wino(s, c, x, u, bias, res, y, ws, st); }, st, ev.e0,
                            ev.e1, &us);
            if (e != hipSuccess) break;
            if (us < best_us) {
                best_us = us;
                best = c;
            }
        }
        (void)hipStreamSynchronize(st);
    }
    if (ws) (void)hipFree(ws);
    if (e != hipSuccess) return hip_fail(e, "Winograd tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_wino_db[key] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

namespace {
GroupKey i8_key(const ConvShape& s, int out) {
    return {device_arch(), {s.N, s.C, s.H, s.W, s.K, s.R, s.S, s.sh, s.sw, s.ph, s.pw, out}};
}
}  // namespace

bool tuned_int8_config(const ConvShape& s, int out, ConvConfig* cfg) {
    const GroupKey key = i8_key(s, out);
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_i8_db.find(key);
    if (it == g_i8_db.end() || !int8_config_valid(s, it->second.cfg)) return false;
    *cfg = it->second.cfg;
    return true;
}

// Every valid integer-conv configuration, timed with the caller's buffers
// (their contents do not change the time); keeps the fastest with its time.
int tune_int8(const I8Member& m, hipStream_t st, ConvConfig* best_out, float* us_out) {
    const ConvShape& s = m.s;
    const int out = m.yq ? (m.y ? 3 : 2) : 0;
    const GroupKey key = i8_key(s, out);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_i8_db.find(key);
        if (it != g_i8_db.end() && int8_config_valid(s, it->second.cfg)) {
            *best_out = it->second.cfg;
            if (us_out) *us_out = it->second.us;
            return NEO_OK;
        }
    }
    ConvConfig best = choose_int8_config(s);
    float best_us = 1e30f;
    hipError_t e = hipSuccess;
    {
        Events ev;
        for (int fk : {1, 2, 4, 8})
            for (int fp : {1, 2, 4})
                for (int wv : {1, 2, 4}) {
                    const ConvConfig c{fk, fp, 1, wv};
                    if (!int8_config_valid(s, c)) continue;
                    float us = 0.f;
                    e = time_launch([&] { return launch_conv_int8_m(m, c, st); },
                                    st, ev.e0, ev.e1, &us);
                    if (e != hipSuccess) break;
                    if (us < best_us) {
                        best_us = us;
                        best = c;
                    }
                }
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "int8 tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_i8_db[key] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

namespace {
// the shape of an integer conv from its key ints (N C H W K R S sh sw ph pw
// ...), or false when they name no convolution
bool i8_shape(const int* q, ConvShape* cs) {
    if (!(q[0] > 0 && q[1] > 0 && q[2] > 0 && q[3] > 0 && q[4] > 0 && q[5] > 0 && q[6] > 0 && q[7] > 0 &&
          q[8] > 0 && q[9] >= 0 && q[10] >= 0))
        return false;
    const int OH = (q[2] + 2 * q[9] - q[5]) / q[7] + 1, OW = (q[3] + 2 * q[10] - q[6]) / q[8] + 1;
    *cs = ConvShape{q[0], q[1], q[2], q[3], q[4], q[5], q[6], q[7], q[8], q[9], q[10], OH, OW, 0, 0, 0};
    return OH > 0 && OW > 0;
}
}  // namespace

// Every configuration valid for all members of an integer group, timed with
// the caller's buffers; keeps the fastest with its time.
int tune_int8_group(const I8Member* m, int n, const GroupPool* pool, hipStream_t st, ConvConfig* best_out,
                    float* us_out) {
    // key: n, m (0 or 1 pools), the members' shapes and output modes, the pool's
    if (n < 1 || n > kMaxGroupConvs) return fail(NEO_ERR_INVALID_ARG, "int8 group tuning: 1 to 4 members");
    GroupKey key{device_arch(), {n, pool ? 1 : 0}};
    ConvShape shp[kMaxGroupConvs];
    for (int i = 0; i < n; ++i) {
        const ConvShape& c = m[i].s;
        shp[i] = c;
        const int out = m[i].yq ? (m[i].y ? 3 : 2) : 0;
        key.second.insert(key.second.end(), {c.N, c.C, c.H, c.W, c.K, c.R, c.S, c.sh, c.sw, c.ph, c.pw, out});
    }
    if (pool) {  // the pool's shape and its output mode (0 float32, 2 int8, 3 both)
        const std::vector<int> pi = pool_ints(*pool);
        key.second.insert(key.second.end(), pi.begin(), pi.end());
        key.second.push_back(pool->q.yq ? (pool->y ? 3 : 2) : 0);
    }
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_i8group_db.find(key);
        if (it != g_i8group_db.end() && int8_group_config_valid(shp, n, it->second.cfg)) {
            *best_out = it->second.cfg;
            if (us_out) *us_out = it->second.us;
            return NEO_OK;
        }
    }
    ConvConfig best = choose_int8_group_config(shp, n);
    float best_us = 1e30f;
    hipError_t e = hipSuccess;
    {
        Events ev;
        for (int fk : {1, 2, 4, 8})
            for (int fp : {1, 2, 4})
                for (int wv : {1, 2, 4}) {
                    const ConvConfig c{fk, fp, 1, wv};
                    if (e != hipSuccess || !int8_group_config_valid(shp, n, c)) continue;
                    float us = 0.f;
                    e = time_launch([&] { return launch_conv_int8_group(m, n, c, pool, st); }, st, ev.e0,
                                    ev.e1, &us);
                    if (e == hipSuccess && us < best_us) {
                        best_us = us;
                        best = c;
                    }
                }
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "int8 group tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_i8group_db[key] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

int tune_conv_group(const ConvShape* s, int n, const float* const* x, const float* const* w,
                    const float* const* bias, const float* const* res, float* const* y,
                    const GroupPool* pool, hipStream_t st, ConvConfig* best_out, float* us_out) {
    GroupKey key{device_arch(), {}};
    for (int i = 0; i < n; ++i)
        key.second.insert(key.second.end(), {s[i].N, s[i].C, s[i].H, s[i].W, s[i].K, s[i].R, s[i].S,
                                             s[i].sh, s[i].sw, s[i].ph, s[i].pw});
    if (pool) {
        const std::vector<int> pi = pool_ints(*pool);
        key.second.insert(key.second.end(), pi.begin(), pi.end());
    }
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_group_db.find(key);
        if (it != g_group_db.end()) {
            *best_out = it->second.cfg;
            if (us_out) *us_out = it->second.us;
            return NEO_OK;
        }
    }
    ConvConfig best = choose_group_config(s, n);
    float best_us = 1e30f;
    hipError_t e = hipSuccess;
    {
        Events ev;
        for (int fk : {1, 2, 4})
            for (int fp : {1, 2, 4})
                for (int wv : {1, 2, 4, 8, 16}) {
                    const ConvConfig c{fk, fp, 1, wv};
                    if (e != hipSuccess || !conv_group_config_valid(s, n, c)) continue;
                    float us = 0.f;
                    e = time_launch([&] { return launch_conv_group(s, n, c, x, w, bias, res, y, pool, st); },
                                    st, ev.e0, ev.e1, &us);
                    if (e == hipSuccess && us < best_us) {
                        best_us = us;
                        best = c;
                    }
                }
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "group tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_group_db[key] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

int tune_conv_pair(const ConvShape& a, const ConvShape& b, const float* x, const float* wa,
                   const float* ba, const float* res, float* y, const float* wb, const float* bb,
                   float* z, hipStream_t st, float* us_out) {
    GroupKey key{device_arch(), {}};
    for (const ConvShape* s : {&a, &b})
        key.second.insert(key.second.end(), {s->N, s->C, s->H, s->W, s->K, s->R, s->S, s->sh, s->sw,
                                             s->ph, s->pw});
    key.second.push_back(res ? 1 : 0);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_pair_db.find(key);
        if (it != g_pair_db.end()) {
            *us_out = it->second;
            return NEO_OK;
        }
    }
    float us = 0.f;
    hipError_t e;
    {
        Events ev;
        e = time_launch([&] { return launch_conv_pair(a, b, x, wa, ba, res, y, wb, bb, z, st); }, st,
                        ev.e0, ev.e1, &us);
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "pair timing");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_pair_db[key] = us;
    }
    *us_out = us;
    return NEO_OK;
}

int tune_conv_chain(const ConvShape* s, int n, const float* x, const float* w0, const float* b0,
                    const float* wa, const float* ba, const float* res, float* y, const float* wb,
                    const float* bb, float* z, hipStream_t st, float* us_out) {
    GroupKey key{device_arch(), {}};
    for (int m = 0; m < n; ++m)
        key.second.insert(key.second.end(), {s[m].N, s[m].C, s[m].H, s[m].W, s[m].K, s[m].R, s[m].S,
                                             s[m].sh, s[m].sw, s[m].ph, s[m].pw});
    key.second.push_back(res ? 1 : 0);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_chain_db.find(key);
        if (it != g_chain_db.end()) {
            *us_out = it->second;
            return NEO_OK;
        }
    }
    float us = 0.f;
    hipError_t e;
    {
        Events ev;
        e = time_launch([&] { return launch_conv_chain(s, n, x, w0, b0, wa, ba, res, y, wb, bb, z, st); },
                        st, ev.e0, ev.e1, &us);
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "chain timing");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_chain_db[key] = us;
    }
    *us_out = us;
    return NEO_OK;
}

int tune_conv_pool(const ConvShape& c, const PoolShape& p, const float* x, const float* w,
                   const float* bias, float* y, hipStream_t st, ConvPoolConfig* best_out,
                   float* us_out) {
    GroupKey key{device_arch(), {c.N, c.C, c.H, c.W, c.K, c.R, c.S, c.sh, c.sw, c.ph, c.pw, c.xb,
                                 c.act}};
    const std::vector<int> pk = pool_ints(GroupPool{p, true, nullptr, nullptr});
    key.second.insert(key.second.end(), pk.begin(), pk.end());
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_convpool_db.find(key);
        if (it != g_convpool_db.end()) {
            *best_out = it->second.cfg;
            *us_out = it->second.us;
            return NEO_OK;
        }
    }
    ConvPoolConfig best = choose_conv_pool_config(c, p);
    float best_us = 1e30f;
    hipError_t e = hipSuccess;
    {
        Events ev;
        for (const ConvPoolConfig& k : conv_pool_candidates(c, p)) {
            float us = 0.f;
            e = time_launch([&] { return launch_conv_pool(c, p, k, x, w, bias, y, st); }, st, ev.e0,
                            ev.e1, &us);
            if (e != hipSuccess) break;
            if (us < best_us) {
                best_us = us;
                best = k;
            }
        }
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "conv-pool tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_convpool_db[key] = PoolEntry{best, best_us};
    }
    *best_out = best;
    *us_out = best_us;
    return NEO_OK;
}

int tune_pool(const GroupPool& p, hipStream_t st, float* us_out) {
    if (p.q.yq) {
        // a pool writing an int8 copy (its float32 output may be absent):
        // timed as it runs, not kept (the results file keys pools by shape)
        float us = 0.f;
        hipError_t e;
        {
            Events ev;
            e = time_launch([&] { return launch_pool_q(p.s, p.max, p.x, p.y, p.q, st); }, st, ev.e0, ev.e1,
                            &us);
            (void)hipStreamSynchronize(st);
        }
        if (e != hipSuccess) return hip_fail(e, "pool timing");
        *us_out = us;
        return NEO_OK;
    }
    const GroupKey key{device_arch(), pool_ints(p)};
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_pool_db.find(key);
        if (it != g_pool_db.end()) {
            *us_out = it->second;
            return NEO_OK;
        }
    }
    float us = 0.f;
    hipError_t e;
    {
        Events ev;
        e = time_launch([&] { return p.max ? launch_maxpool(p.s, p.x, p.y, st) : launch_avgpool(p.s, p.x, p.y, st); },
                        st, ev.e0, ev.e1, &us);
        (void)hipStreamSynchronize(st);
    }
    if (e != hipSuccess) return hip_fail(e, "pool timing");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_pool_db[key] = us;
    }
    *us_out = us;
    return NEO_OK;
}

}  // namespace neo

using namespace neo;

extern "C" {

// Text format, one workload per line:
//   arch N C H W K R S sh sw ph pw wmfma xb yb fk fp split waves us
// one line per fused launch of n NCHW16c convs and m (0 or 1) pooling steps:
//   group arch n m (N C H W K R S sh sw ph pw) x n (max N C H W R S sh sw ph pw xb) x m
//         fk fp split waves us
// one line per pooling step timed alone:
//   pool arch max N C H W R S sh sw ph pw xb us
// one line per pair of pointwise convs in one launch:
//   pair arch (N C H W K R S sh sw ph pw) x 2 residual us
// one line per 3x3-led chain of n (2 or 3) convs in one launch:
//   chain arch n (N C H W K R S sh sw ph pw) x n residual us
// one line per stem conv with its max pooling in one launch:
//   convpool arch N C H W K R S sh sw ph pw xb act (max N C H W R S sh sw ph pw xb)
//            fk fp waves ty tx us
// one line per 3x3 stride-1 conv by Winograd F(2x2, 3x3):
//   wino arch N C H W K ph pw fk fp split waves us
// one line per integer conv (out: 0 float32, 2 int8, 3 both outputs):
//   int8 arch N C H W K R S sh sw ph pw out fk fp waves us
// and one line per launch of n integer convs and m (0 or 1) pooling steps:
//   i8group arch n m (N C H W K R S sh sw ph pw out) x n (max N C H W R S sh sw ph pw xb out) x m
//           fk fp waves us
int neo_tune_db_save(const char* path) {
    if (!path) return fail(NEO_ERR_INVALID_ARG, "neo_tune_db_save: path is NULL");
    std::ofstream f(path);
    if (!f) return fail(NEO_ERR_INVALID_ARG, std::string("neo_tune_db_save: cannot open ") + path);
    std::lock_guard<std::mutex> lk(g_mu);
    f.precision(9);  // times round-trip exactly, so a reload makes the same choices
    for (const auto& kv : g_db) {
        const Key& k = kv.first;
        const Entry& v = kv.second;
        f << k.arch << ' ' << k.N << ' ' << k.C << ' ' << k.H << ' ' << k.W << ' ' << k.K << ' ' << k.R
          << ' ' << k.S << ' ' << k.sh << ' ' << k.sw << ' ' << k.ph << ' ' << k.pw << ' ' << k.wmfma
          << ' ' << k.xb << ' ' << k.yb << ' ' << v.cfg.fk << ' ' << v.cfg.fp << ' ' << v.cfg.split
          << ' ' << v.cfg.waves << ' ' << v.us << '\n';
    }
    for (const auto& kv : g_group_db) {
        const std::vector<int>& k = kv.first.second;
        const Entry& v = kv.second;
        // 11 n + 12 m ints with n <= 4, m <= 1: m is the remainder's sign
        const size_t m = k.size() % kGroupShapeInts ? 1 : 0;
        f << "group " << kv.first.first << ' ' << (k.size() - m * kPoolShapeInts) / kGroupShapeInts
          << ' ' << m;
        for (int x : k) f << ' ' << x;
        f << ' ' << v.cfg.fk << ' ' << v.cfg.fp << ' ' << v.cfg.split << ' ' << v.cfg.waves << ' '
          << v.us << '\n';
    }
    for (const auto* db : {&g_pool_db, &g_pair_db}) {
        for (const auto& kv : *db) {
            f << (db == &g_pool_db ? "pool " : "pair ") << kv.first.first;
            for (int x : kv.first.second) f << ' ' << x;
            f << ' ' << kv.second << '\n';
        }
    }
    for (const auto& kv : g_chain_db) {
        f << "chain " << kv.first.first << ' ' << kv.first.second.size() / kGroupShapeInts;
        for (int x : kv.first.second) f << ' ' << x;
        f << ' ' << kv.second << '\n';
    }
    for (const auto& kv : g_convpool_db) {
        f << "convpool " << kv.first.first;
        for (int x : kv.first.second) f << ' ' << x;
        const ConvPoolConfig& c = kv.second.cfg;
        f << ' ' << c.fk << ' ' << c.fp << ' ' << c.waves << ' ' << c.ty << ' ' << c.tx << ' '
          << kv.second.us << '\n';
    }
    for (const auto& kv : g_wino_db) {
        f << "wino " << kv.first.first;
        for (int x : kv.first.second) f << ' ' << x;
        const ConvConfig& c = kv.second.cfg;
        f << ' ' << c.fk << ' ' << c.fp << ' ' << c.split << ' ' << c.waves << ' ' << kv.second.us << '\n';
    }
    for (const auto& kv : g_i8_db) {
        f << "int8 " << kv.first.first;
        for (int x : kv.first.second) f << ' ' << x;
        const ConvConfig& c = kv.second.cfg;
        f << ' ' << c.fk << ' ' << c.fp << ' ' << c.waves << ' ' << kv.second.us << '\n';
    }
    for (const auto& kv : g_i8group_db) {
        f << "i8group " << kv.first.first;  // the key's ints start with n and m
        for (int x : kv.first.second) f << ' ' << x;
        const ConvConfig& c = kv.second.cfg;
        f << ' ' << c.fk << ' ' << c.fp << ' ' << c.waves << ' ' << kv.second.us << '\n';
    }
    return f ? (int)(g_db.size() + g_group_db.size() + g_pool_db.size() + g_pair_db.size() +
                     g_chain_db.size() + g_convpool_db.size() + g_wino_db.size() + g_i8_db.size() +
                     g_i8group_db.size())
             : fail(NEO_ERR_INVALID_ARG, "neo_tune_db_save: write failed");
}

int neo_tune_db_load(const char* path) {
    if (!path) return fail(NEO_ERR_INVALID_ARG, "neo_tune_db_load: path is NULL");
    std::ifstream f(path);
    if (!f) return fail(NEO_ERR_INVALID_ARG, std::string("neo_tune_db_load: cannot open ") + path);
    std::string line;
    int n = 0, lineno = 0;
    std::map<Key, Entry> add;
    std::map<GroupKey, Entry> add_group;
    std::map<GroupKey, float> add_pool, add_pair, add_chain;
    std::map<GroupKey, PoolEntry> add_convpool;
    std::map<GroupKey, Entry> add_wino, add_i8, add_i8group;
    auto read_ints = [](std::istringstream& is, int count, std::vector<int>& out) {
        for (int i = 0; i < count; ++i) {
            int x = 0;
            if (!(is >> x)) return false;
            out.push_back(x);
        }
        return true;
    };
    const std::string bad = "neo_tune_db_load: malformed line ";
    while (std::getline(f, line)) {
        ++lineno;
        if (line.empty() || line[0] == '#') continue;
        std::istringstream is(line);
        Key k;
        Entry v;
        if (line.compare(0, 6, "group ") == 0) {
            std::string tag;
            GroupKey gk;
            int members = 0, pools = -1;
            bool ok = (bool)(is >> tag >> gk.first >> members >> pools) && members >= 1 &&
                      members <= kMaxGroupConvs && (pools == 0 || pools == 1);
            ok = ok && read_ints(is, members * kGroupShapeInts + pools * kPoolShapeInts, gk.second);
            ok = ok && (is >> v.cfg.fk >> v.cfg.fp >> v.cfg.split >> v.cfg.waves >> v.us) &&
                 v.cfg.split == 1 && conv_config_valid(v.cfg);
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_group[gk] = v;
            ++n;
            continue;
        }
        if (line.compare(0, 5, "pair ") == 0) {
            std::string tag;
            GroupKey pk;
            float us = 0.f;
            const bool ok = (bool)(is >> tag >> pk.first) && read_ints(is, kPairInts, pk.second) &&
                            (bool)(is >> us);
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_pair[pk] = us;
            ++n;
            continue;
        }
        if (line.compare(0, 6, "chain ") == 0) {
            std::string tag;
            GroupKey ck;
            int convs = 0;
            float us = 0.f;
            const bool ok = (bool)(is >> tag >> ck.first >> convs) && (convs == 2 || convs == 3) &&
                            read_ints(is, convs * kGroupShapeInts + 1, ck.second) && (bool)(is >> us);
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_chain[ck] = us;
            ++n;
            continue;
        }
        if (line.compare(0, 9, "convpool ") == 0) {
            std::string tag;
            GroupKey ck;
            PoolEntry pe;
            bool ok = (bool)(is >> tag >> ck.first) && read_ints(is, kConvPoolInts, ck.second) &&
                      (bool)(is >> pe.cfg.fk >> pe.cfg.fp >> pe.cfg.waves >> pe.cfg.ty >> pe.cfg.tx >>
                             pe.us);
            if (ok) {  // the entry must name a configuration the kernel takes for its shapes
                const std::vector<int>& v = ck.second;
                ConvShape cs{v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7], v[8], v[9], v[10],
                             (v[2] + 2 * v[9] - v[5]) / v[7] + 1, (v[3] + 2 * v[10] - v[6]) / v[8] + 1,
                             0, 0, v[12]};
                cs.xb = v[11];
                cs.yb = 16;
                PoolShape ps{v[14], v[15], v[16], v[17], v[18], v[19], v[20], v[21], v[22], v[23],
                             0, 0, 0, 0};
                ps.OH = (ps.H + 2 * ps.ph - ps.R) / ps.sh + 1;
                ps.OW = (ps.W + 2 * ps.pw - ps.S) / ps.sw + 1;
                ps.xb = v[24];
                ok = v[7] > 0 && v[8] > 0 && ps.sh > 0 && ps.sw > 0 &&
                     conv_pool_config_valid(cs, ps, pe.cfg);
            }
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_convpool[ck] = pe;
            ++n;
            continue;
        }
        if (line.compare(0, 5, "wino ") == 0) {
            std::string tag;
            GroupKey wk;
            bool ok = (bool)(is >> tag >> wk.first) && read_ints(is, kWinoInts, wk.second) &&
                      (bool)(is >> v.cfg.fk >> v.cfg.fp >> v.cfg.split >> v.cfg.waves >> v.us);
            if (ok) {  // the entry must name a configuration the kernel takes for its shape
                const std::vector<int>& q = wk.second;
                ConvShape cs{q[0], q[1], q[2], q[3], q[4], 3, 3, 1, 1, q[5], q[6],
                             q[2] + 2 * q[5] - 2, q[3] + 2 * q[6] - 2, 0, 0, 0};
                ok = q[0] > 0 && q[1] > 0 && q[2] > 0 && q[3] > 0 && q[4] > 0 && q[5] >= 0 &&
                     q[6] >= 0 && wino_config_valid(cs, v.cfg);
            }
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_wino[wk] = v;
            ++n;
            continue;
        }
        if (line.compare(0, 5, "int8 ") == 0) {
            std::string tag;
            GroupKey ik;
            v.cfg.split = 1;
            bool ok = (bool)(is >> tag >> ik.first) && read_ints(is, kI8Ints, ik.second) &&
                      (bool)(is >> v.cfg.fk >> v.cfg.fp >> v.cfg.waves >> v.us);
            if (ok) {  // the entry must name a configuration the kernel takes for its shape
                const std::vector<int>& q = ik.second;
                ok = q[0] > 0 && q[1] > 0 && q[2] > 0 && q[3] > 0 && q[4] > 0 && q[5] > 0 && q[6] > 0 &&
                     q[7] > 0 && q[8] > 0 && q[9] >= 0 && q[10] >= 0 &&
                     (q[11] == 0 || q[11] == 2 || q[11] == 3);
                if (ok) {
                    const int OH = (q[2] + 2 * q[9] - q[5]) / q[7] + 1, OW = (q[3] + 2 * q[10] - q[6]) / q[8] + 1;
                    ConvShape cs{q[0], q[1], q[2], q[3], q[4], q[5], q[6], q[7], q[8], q[9], q[10],
                                 OH, OW, 0, 0, 0};
                    ok = OH > 0 && OW > 0 && int8_config_valid(cs, v.cfg);
                }
            }
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_i8[ik] = v;
            ++n;
            continue;
        }
        if (line.compare(0, 8, "i8group ") == 0) {
            std::string tag;
            GroupKey gk;
            int members = 0, pools = -1;
            v.cfg.split = 1;
            bool ok = (bool)(is >> tag >> gk.first >> members >> pools) && members >= 1 &&
                      members <= kMaxGroupConvs && (pools == 0 || pools == 1);
            if (ok) {
                gk.second = {members, pools};
                ok = read_ints(is, members * kI8Ints + pools * (kPoolShapeInts + 1), gk.second) &&
                     (bool)(is >> v.cfg.fk >> v.cfg.fp >> v.cfg.waves >> v.us);
            }
            ConvShape shp[kMaxGroupConvs];
            for (int i = 0; ok && i < members; ++i) {
                const int* q = gk.second.data() + 2 + i * kI8Ints;
                ok = i8_shape(q, &shp[i]) && (q[11] == 0 || q[11] == 2 || q[11] == 3);
            }
            // the pool rides in blocks of 16 only; its output mode 0, 2 or 3
            const int pm = gk.second.back();
            ok = ok && (pools == 0 || (gk.second[gk.second.size() - 2] == 16 && (pm == 0 || pm == 2 || pm == 3))) &&
                 int8_group_config_valid(shp, members, v.cfg);
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_i8group[gk] = v;
            ++n;
            continue;
        }
        if (line.compare(0, 5, "pool ") == 0) {
            std::string tag;
            GroupKey pk;
            float us = 0.f;
            bool ok = (bool)(is >> tag >> pk.first) && read_ints(is, kPoolShapeInts, pk.second) &&
                      (bool)(is >> us) && pow2_block(pk.second.back());
            if (!ok) return fail(NEO_ERR_INVALID_ARG, bad + std::to_string(lineno));
            add_pool[pk] = us;
            ++n;
            continue;
        }
        if (!(is >> k.arch >> k.N >> k.C >> k.H >> k.W >> k.K >> k.R >> k.S >> k.sh >> k.sw >> k.ph >>
              k.pw >> k.wmfma >> k.xb >> k.yb >> v.cfg.fk >> v.cfg.fp >> v.cfg.split >> v.cfg.waves >>
              v.us) ||
            !conv_any_config_valid(v.cfg) || !key_blocks_valid(k) || (v.cfg.fp == 0 && !k.wmfma))
            return fail(NEO_ERR_INVALID_ARG,
                        "neo_tune_db_load: malformed line " + std::to_string(lineno));
        add[k] = v;
        ++n;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    for (const auto& kv : add) g_db[kv.first] = kv.second;
    for (const auto& kv : add_group) g_group_db[kv.first] = kv.second;
    for (const auto& kv : add_pool) g_pool_db[kv.first] = kv.second;
    for (const auto& kv : add_pair) g_pair_db[kv.first] = kv.second;
    for (const auto& kv : add_chain) g_chain_db[kv.first] = kv.second;
    for (const auto& kv : add_convpool) g_convpool_db[kv.first] = kv.second;
    for (const auto& kv : add_wino) g_wino_db[kv.first] = kv.second;
    for (const auto& kv : add_i8) g_i8_db[kv.first] = kv.second;
    for (const auto& kv : add_i8group) g_i8group_db[kv.first] = kv.second;
    return n;
}

void neo_tune_db_clear(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_db.clear();
    g_group_db.clear();
    g_pool_db.clear();
    g_pair_db.clear();
    g_chain_db.clear();
    g_convpool_db.clear();
    g_wino_db.clear();
    g_i8_db.clear();
    g_i8group_db.clear();
}

int neo_tune_db_size(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return (int)(g_db.size() + g_group_db.size() + g_pool_db.size() + g_pair_db.size() +
                 g_chain_db.size() + g_convpool_db.size() + g_wino_db.size() + g_i8_db.size() +
                 g_i8group_db.size());
}

}  // extern "C"
