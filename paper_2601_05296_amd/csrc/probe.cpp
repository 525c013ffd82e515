// probe.cpp -- optional per-kernel timing. While enabled, every entry point
// records a start event on its stream and one event after each kernel it
// launches; the elapsed time between consecutive events of one call is the
// duration of the kernel in between. Disabled (the default) it costs one
// branch per launch. Not thread-safe: enable it from a single host thread.
#include <hip/hip_runtime.h>

#include <vector>

#include "probe.hpp"

namespace moe {
namespace probe {
namespace {

struct Rec {
    const char* name;  // nullptr for the start event of a call
    hipEvent_t ev;
};

bool g_on = false;
std::vector<hipEvent_t> g_pool;
std::vector<Rec> g_recs;
int g_dropped = 0;   // records not taken because the events ran out

void record(const char* name, hipStream_t st) {
    if (g_recs.size() >= g_pool.size()) {   // capacity reached: count, do not record
        ++g_dropped;
        return;
    }
    hipEvent_t ev = g_pool[g_recs.size()];
    if (hipEventRecord(ev, st) != hipSuccess) return;
    g_recs.push_back(Rec{name, ev});
}

}  // namespace

bool enabled() { return g_on; }
void begin(hipStream_t st) { if (g_on) record(nullptr, st); }
void mark(const char* name, hipStream_t st) { if (g_on) record(name, st); }

int enable(int capacity) {
    disable();
    g_pool.resize(capacity);
    for (int i = 0; i < capacity; ++i)
        if (hipEventCreate(&g_pool[i]) != hipSuccess) {
            g_pool.resize(i);
            disable();
            return -1;
        }
    g_recs.reserve(capacity);
    g_dropped = 0;
    g_on = true;
    return 0;
}

void disable() {
    g_on = false;
    for (hipEvent_t e : g_pool) (void)hipEventDestroy(e);
    g_pool.clear();
    g_recs.clear();
    g_dropped = 0;
}

int dropped() { return g_dropped; }

int count() {
    int n = 0;
    for (const Rec& r : g_recs) n += r.name != nullptr;
    return n;
}

int get(int i, const char** name, float* ms) {
    int n = -1;
    for (size_t j = 0; j < g_recs.size(); ++j) {
        if (!g_recs[j].name) continue;
        if (++n != i) continue;
        if (j == 0) return -1;
        *name = g_recs[j].name;
        if (hipEventSynchronize(g_recs[j].ev) != hipSuccess) return -1;
        return hipEventElapsedTime(ms, g_recs[j - 1].ev, g_recs[j].ev) == hipSuccess ? 0 : -1;
    }
    return -1;
}

}  // namespace probe
}  // namespace moe
