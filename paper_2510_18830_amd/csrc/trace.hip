// Kernel-level tracing (see trace.h).
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/msparse.h"
#include "trace.h"

namespace msparse {

namespace {

struct Rec {
    const char* name;
    hipEvent_t start, stop;
};

std::mutex g_mu;
bool g_on = false;
std::vector<Rec> g_open;    // begun, not ended (per-thread nesting is not needed: launches are sequential)
std::vector<Rec> g_done;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

}  // namespace

bool trace_on() {
    std::lock_guard<std::mutex> lk(g_mu);
    return g_on;
}

void trace_begin(const char* name, hipStream_t s) {
    std::lock_guard<std::mutex> lk(g_mu);
    Rec r{name, take_event(), take_event()};
    if (r.start) (void)hipEventRecord(r.start, s);
    g_open.push_back(r);
}

void trace_end(hipStream_t s) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_open.empty()) return;
    Rec r = g_open.back();
    g_open.pop_back();
    if (r.stop) (void)hipEventRecord(r.stop, s);
    g_done.push_back(r);
}

}  // namespace msparse

using namespace msparse;

extern "C" {

void msparse_trace_enable(int32_t on) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_on = on != 0;
}

int32_t msparse_trace_read(msparse_trace_entry* out, int32_t cap) {
    std::vector<Rec> done;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        done.swap(g_done);
    }
    std::vector<msparse_trace_entry> agg;
    for (const Rec& r : done) {
        float ms = 0.f;
        if (r.stop) (void)hipEventSynchronize(r.stop);
        if (r.start && r.stop && hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) ms = 0.f;
        size_t i = 0;
        for (; i < agg.size(); ++i)
            if (std::strcmp(agg[i].name, r.name) == 0) break;
        if (i == agg.size()) {
            msparse_trace_entry e{};
            std::strncpy(e.name, r.name, sizeof(e.name) - 1);
            agg.push_back(e);
        }
        agg[i].launches += 1;
        agg[i].total_ms += ms;
    }
    {
        std::lock_guard<std::mutex> lk(g_mu);
        for (const Rec& r : done) {
            if (r.start) g_pool.push_back(r.start);
            if (r.stop) g_pool.push_back(r.stop);
        }
    }
    const int32_t n = int32_t(agg.size());
    for (int32_t i = 0; i < n && i < cap; ++i) out[i] = agg[i];
    return n;
}

}  // extern "C"
