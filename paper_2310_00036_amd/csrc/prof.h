// Optional per-launch kernel timing with HIP events on the launching stream, used by the
// benchmark to measure a kernel's average duration inside a timed region. Off by default:
// a disabled scope costs one branch.
#pragma once

#include <hip/hip_runtime.h>

#include <string>

namespace cb {

bool prof_active();
// Returns a slot to close with prof_end(), or -1 when this launch is not recorded.
int prof_begin(const std::string& key, hipStream_t s);
void prof_end(int slot, hipStream_t s);

// RAII helper: records around the launches in its scope when profiling is active.
struct ProfScope {
    int slot = -1;
    hipStream_t stream;
    template <class KeyFn>
    ProfScope(hipStream_t s, KeyFn key) : stream(s) {
        if (prof_active()) slot = prof_begin(key(), s);
    }
    ~ProfScope() {
        if (slot >= 0) prof_end(slot, stream);
    }
};

}  // namespace cb
