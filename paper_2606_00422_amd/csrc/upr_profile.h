// RAII timing scope around one kernel launch (see upr_profile.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "upr.h"

namespace upr {

class ProfScope {
public:
    ProfScope(const char* name, hipStream_t s);
    ~ProfScope();
    ProfScope(const ProfScope&) = delete;
    ProfScope& operator=(const ProfScope&) = delete;

private:
    hipStream_t stream_;
    int64_t index_ = -1;
};

}  // namespace upr
