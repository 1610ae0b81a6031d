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

}  // namespace

bool tuned_config(const ConvShape& s, bool wmfma, ConvConfig* out) {
    const std::string arch = device_arch();
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_db.find(key_of(s, wmfma, arch));
    if (it == g_db.end()) return false;
    *out = it->second.cfg;
    return true;
}

// Time every candidate on `st` (a stream that is not the legacy null stream)
// with the caller's buffers: each candidate's launches are captured into a
// graph of `reps` launches and replayed between two events.  Keeps the
// fastest in the database and returns it with its time per launch (us_out may
// be null).
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
    const std::vector<ConvConfig> cands = candidates(s);
    size_t ws_bytes = 0;
    for (const ConvConfig& c : cands) ws_bytes = std::max(ws_bytes, conv_workspace_bytes(s, c));
    float* ws = nullptr;
    hipError_t e = hipSuccess;
    if (ws_bytes) e = hipMalloc(&ws, ws_bytes);
    if (e != hipSuccess) return fail(NEO_ERR_OOM, "tuning workspace allocation");
    hipEvent_t e0, e1;
    (void)hipEventCreate(&e0);
    (void)hipEventCreate(&e1);
    const int reps = 10;
    ConvConfig best = choose_conv_config(s);
    float best_us = 1e30f;
    int rc = NEO_OK;
    for (const ConvConfig& c : cands) {
        // warm-up launch (also surfaces a launch error before capture)
        e = launch_conv2d(s, c, x, w, wmfma, bias, res, y, ws, st);
        if (e != hipSuccess) {
            rc = hip_fail(e, "tuning launch");
            break;
        }
        hipGraph_t g = nullptr;
        hipGraphExec_t ge = nullptr;
        e = hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal);
        for (int i = 0; i < reps && e == hipSuccess; ++i)
            e = launch_conv2d(s, c, x, w, wmfma, bias, res, y, ws, st);
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
        if (e != hipSuccess) {
            rc = hip_fail(e, "tuning timing");
            break;
        }
        const float us = ms * 1000.f / reps;
        if (us < best_us) {
            best_us = us;
            best = c;
        }
    }
    (void)hipStreamSynchronize(st);
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (ws) (void)hipFree(ws);
    if (rc != NEO_OK) return rc;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_db[key_of(s, wmfma, arch)] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

namespace {
// one launch of several convs: architecture and the members' shapes -> config
using GroupKey = std::pair<std::string, std::vector<int>>;
std::map<GroupKey, Entry> g_group_db;
constexpr int kGroupShapeInts = 11;  // N C H W K R S sh sw ph pw per member
}

int tune_conv_group(const ConvShape* s, int n, const float* const* x, const float* const* w,
                    const float* const* bias, const float* const* res, float* const* y,
                    hipStream_t st, ConvConfig* best_out, float* us_out) {
    GroupKey key{device_arch(), {}};
    for (int i = 0; i < n; ++i)
        key.second.insert(key.second.end(), {s[i].N, s[i].C, s[i].H, s[i].W, s[i].K, s[i].R, s[i].S,
                                             s[i].sh, s[i].sw, s[i].ph, s[i].pw});
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_group_db.find(key);
        if (it != g_group_db.end()) {
            *best_out = it->second.cfg;
            if (us_out) *us_out = it->second.us;
            return NEO_OK;
        }
    }
    hipEvent_t e0, e1;
    (void)hipEventCreate(&e0);
    (void)hipEventCreate(&e1);
    const int reps = 10;
    ConvConfig best = choose_group_config(s, n);
    float best_us = 1e30f;
    hipError_t e = hipSuccess;
    for (int fk : {1, 2, 4})
        for (int fp : {1, 2, 4})
            for (int wv : {1, 2, 4, 8, 16}) {
                const ConvConfig c{fk, fp, 1, wv};
                if (e != hipSuccess || !conv_group_config_valid(s, n, c)) continue;
                e = launch_conv_group(s, n, c, x, w, bias, res, y, st);  // warm-up
                if (e != hipSuccess) break;
                hipGraph_t g = nullptr;
                hipGraphExec_t ge = nullptr;
                e = hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal);
                for (int i = 0; i < reps && e == hipSuccess; ++i)
                    e = launch_conv_group(s, n, c, x, w, bias, res, y, st);
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
                const float us = ms * 1000.f / reps;
                if (e == hipSuccess && us < best_us) {
                    best_us = us;
                    best = c;
                }
            }
    (void)hipStreamSynchronize(st);
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    if (e != hipSuccess) return hip_fail(e, "group tuning");
    {
        std::lock_guard<std::mutex> lk(g_mu);
        g_group_db[key] = Entry{best, best_us};
    }
    *best_out = best;
    if (us_out) *us_out = best_us;
    return NEO_OK;
}

}  // namespace neo

using namespace neo;

extern "C" {

// Text format, one workload per line:
//   arch N C H W K R S sh sw ph pw wmfma xb yb fk fp split waves us
// and one line per fused launch of n NCHW16c convs:
//   group arch n (N C H W K R S sh sw ph pw) x n fk fp split waves us
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
        f << "group " << kv.first.first << ' ' << k.size() / kGroupShapeInts;
        for (int x : k) f << ' ' << x;
        f << ' ' << v.cfg.fk << ' ' << v.cfg.fp << ' ' << v.cfg.split << ' ' << v.cfg.waves << ' '
          << v.us << '\n';
    }
    return f ? (int)(g_db.size() + g_group_db.size())
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
    while (std::getline(f, line)) {
        ++lineno;
        if (line.empty() || line[0] == '#') continue;
        std::istringstream is(line);
        Key k;
        Entry v;
        if (line.compare(0, 6, "group ") == 0) {
            std::string tag;
            GroupKey gk;
            int members = 0;
            bool ok = (bool)(is >> tag >> gk.first >> members) && members >= 1 &&
                      members <= kMaxGroupConvs;
            for (int i = 0; ok && i < members * kGroupShapeInts; ++i) {
                int x = 0;
                ok = (bool)(is >> x);
                gk.second.push_back(x);
            }
            ok = ok && (is >> v.cfg.fk >> v.cfg.fp >> v.cfg.split >> v.cfg.waves >> v.us) &&
                 v.cfg.split == 1 && conv_config_valid(v.cfg);
            if (!ok)
                return fail(NEO_ERR_INVALID_ARG,
                            "neo_tune_db_load: malformed line " + std::to_string(lineno));
            add_group[gk] = v;
            ++n;
            continue;
        }
        if (!(is >> k.arch >> k.N >> k.C >> k.H >> k.W >> k.K >> k.R >> k.S >> k.sh >> k.sw >> k.ph >>
              k.pw >> k.wmfma >> k.xb >> k.yb >> v.cfg.fk >> v.cfg.fp >> v.cfg.split >> v.cfg.waves >>
              v.us) ||
            !conv_config_valid(v.cfg) || !pow2_block(k.xb) || !pow2_block(k.yb))
            return fail(NEO_ERR_INVALID_ARG,
                        "neo_tune_db_load: malformed line " + std::to_string(lineno));
        add[k] = v;
        ++n;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    for (const auto& kv : add) g_db[kv.first] = kv.second;
    for (const auto& kv : add_group) g_group_db[kv.first] = kv.second;
    return n;
}

void neo_tune_db_clear(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_db.clear();
    g_group_db.clear();
}

int neo_tune_db_size(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return (int)(g_db.size() + g_group_db.size());
}

}  // extern "C"
