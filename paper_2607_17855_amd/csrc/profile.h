// Kernel timing hooks (bi_profile_begin / bi_profile_end).
#pragma once

#include <hip/hip_runtime.h>

namespace bi {

bool profiling();
// Record the start (end = false) or the end of a launch of kernel class `name`.
void prof_mark(const char *name, hipStream_t s, bool end);

// Brackets one kernel launch with profiling events when profiling is on.
struct ProfScope {
    const char *name;
    hipStream_t s;
    ProfScope(const char *n, hipStream_t st) : name(n), s(st) { prof_mark(name, s, false); }
    ~ProfScope() { prof_mark(name, s, true); }
};

}  // namespace bi
