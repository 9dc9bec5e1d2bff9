// Kernel-level tracing: when enabled, every internal launch is bracketed by a
// pair of HIP events on its stream; msparse_trace_read sums the durations per
// kernel name.  Off by default (no events, no overhead).
#pragma once

#include <hip/hip_runtime.h>

namespace msparse {

bool trace_on();
void trace_begin(const char* name, hipStream_t s);
void trace_end(hipStream_t s);

struct TraceScope {
    hipStream_t s;
    bool on;
    TraceScope(const char* name, hipStream_t st) : s(st), on(trace_on()) {
        if (on) trace_begin(name, s);
    }
    ~TraceScope() {
        if (on) trace_end(s);
    }
};

}  // namespace msparse
