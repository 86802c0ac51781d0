// Per-launch event timing (see include/cleanba_profile.h).
#include <hip/hip_runtime.h>

#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "../../include/cleanba_profile.h"
#include "prof.h"

namespace cb {
namespace {

struct Rec {
    std::string key;
    int ev;   // index of the start event; ev + 1 is the end event
};

struct Profile {
    bool active = false;
    std::string only;
    std::vector<hipEvent_t> events;
    std::vector<Rec> recs;
    int32_t dropped = 0;
    std::vector<std::string> keys;
    std::vector<double> ms;
    std::vector<int32_t> launches;
};

Profile g;

}  // namespace

bool prof_active() { return g.active; }

int prof_begin(const std::string& key, hipStream_t s) {
    if (!g.only.empty() && key != g.only) return -1;
    const int ev = int(g.recs.size()) * 2;
    if (ev + 1 >= int(g.events.size())) {
        ++g.dropped;
        return -1;
    }
    g.recs.push_back(Rec{key, ev});
    (void)hipEventRecord(g.events[ev], s);
    return ev;
}

void prof_end(int slot, hipStream_t s) { (void)hipEventRecord(g.events[slot + 1], s); }

}  // namespace cb

using namespace cb;

extern "C" {

impala_status_t impala_profile_begin(const char* only_key, int32_t max_launches) {
    if (g.active || max_launches < 1 || max_launches > (1 << 20)) return IMPALA_EINVAL;
    g.only = only_key ? only_key : "";
    g.recs.clear();
    g.keys.clear();
    g.ms.clear();
    g.launches.clear();
    g.dropped = 0;
    g.events.assign(size_t(max_launches) * 2, nullptr);
    for (auto& e : g.events)
        if (hipEventCreate(&e) != hipSuccess) return IMPALA_EHIP;
    g.active = true;
    return IMPALA_OK;
}

int impala_profile_end(void) {
    if (!g.active) return IMPALA_EINVAL;
    g.active = false;
    std::map<std::string, size_t> index;
    for (const Rec& r : g.recs) {
        float ms = 0.f;
        if (hipEventSynchronize(g.events[r.ev + 1]) != hipSuccess ||
            hipEventElapsedTime(&ms, g.events[r.ev], g.events[r.ev + 1]) != hipSuccess)
            return IMPALA_EHIP;
        auto it = index.find(r.key);
        if (it == index.end()) {
            it = index.emplace(r.key, g.keys.size()).first;
            g.keys.push_back(r.key);
            g.ms.push_back(0.0);
            g.launches.push_back(0);
        }
        g.ms[it->second] += ms;
        g.launches[it->second] += 1;
    }
    for (auto& e : g.events) (void)hipEventDestroy(e);
    g.events.clear();
    g.recs.clear();
    return int(g.keys.size());
}

impala_status_t impala_profile_key(int32_t i, char* key, size_t key_cap, double* total_ms,
                                   int32_t* launches) {
    if (i < 0 || size_t(i) >= g.keys.size()) return IMPALA_EINVAL;
    if (key && key_cap) {
        std::strncpy(key, g.keys[i].c_str(), key_cap - 1);
        key[key_cap - 1] = 0;
    }
    if (total_ms) *total_ms = g.ms[i];
    if (launches) *launches = g.launches[i];
    return IMPALA_OK;
}

int32_t impala_profile_dropped(void) { return g.dropped; }

}  // extern "C"
