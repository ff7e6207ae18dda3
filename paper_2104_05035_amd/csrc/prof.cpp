// Opt-in per-kernel timing (see prof.hpp) and its C ABI.
#include <mutex>
#include <string>
#include <vector>

#include "prof.hpp"

namespace rat3d {
namespace {

struct Launch {
    hipEvent_t a, b;
};

struct Tag {
    std::string name;
    int64_t launches = 0;
    double flops = 0.0, bytes = 0.0, ms = 0.0;
    std::vector<Launch> pending;
};

std::mutex g_mu;
bool g_on = false;
std::string g_filter;  // empty: every tag
std::vector<Tag> g_tags;
std::vector<hipEvent_t> g_free;

hipEvent_t get_event() {
    if (!g_free.empty()) {
        hipEvent_t e = g_free.back();
        g_free.pop_back();
        return e;
    }
    // timing only: no system-scope fence on record (no cache writeback and
    // invalidation around every bracketed launch; the host reads only the
    // timestamps)
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

// Waits for a tag's pending launches and folds their durations in.
void settle(Tag& t) {
    for (Launch& l : t.pending) {
        float ms = 0.f;
        if (hipEventSynchronize(l.b) == hipSuccess && hipEventElapsedTime(&ms, l.a, l.b) == hipSuccess)
            t.ms += ms;
        g_free.push_back(l.a);
        g_free.push_back(l.b);
    }
    t.pending.clear();
}

}  // namespace

bool prof_on() { return g_on; }

int prof_begin(const char* tag, hipStream_t st) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_filter.empty() && g_filter != tag) return -1;
    int slot = -1;
    for (size_t i = 0; i < g_tags.size(); ++i)
        if (g_tags[i].name == tag) slot = (int)i;
    if (slot < 0) {
        g_tags.push_back(Tag{});
        g_tags.back().name = tag;
        slot = (int)g_tags.size() - 1;
    }
    hipEvent_t a = get_event(), b = get_event();
    if (!a || !b) return -1;
    hipEventRecord(a, st);
    g_tags[slot].pending.push_back(Launch{a, b});
    return slot;
}

void prof_end(int slot, hipStream_t st, double alg_flops, double alg_bytes) {
    std::lock_guard<std::mutex> lk(g_mu);
    Tag& t = g_tags[slot];
    hipEventRecord(t.pending.back().b, st);
    t.launches += 1;
    t.flops += alg_flops;
    t.bytes += alg_bytes;
    if (t.pending.size() > 4096) settle(t);
}

}  // namespace rat3d

using namespace rat3d;

extern "C" {

rat3d_status rat3d_profile_enable(int enable) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_on = enable != 0;
    return RAT3D_OK;
}

rat3d_status rat3d_profile_filter(const char* tag) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_filter = tag ? tag : "";
    return RAT3D_OK;
}

rat3d_status rat3d_profile_reset(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    for (Tag& t : g_tags) settle(t);
    g_tags.clear();
    return RAT3D_OK;
}

int rat3d_profile_count(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    return (int)g_tags.size();
}

rat3d_status rat3d_profile_read(int i, const char** name, int64_t* launches, double* total_ms,
                                double* alg_flops, double* alg_bytes) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (i < 0 || i >= (int)g_tags.size()) {
        set_error("rat3d_profile_read: index out of range");
        return RAT3D_EINVAL;
    }
    Tag& t = g_tags[i];
    settle(t);
    if (name) *name = t.name.c_str();
    if (launches) *launches = t.launches;
    if (total_ms) *total_ms = t.ms;
    if (alg_flops) *alg_flops = t.flops;
    if (alg_bytes) *alg_bytes = t.bytes;
    return RAT3D_OK;
}

}  // extern "C"
