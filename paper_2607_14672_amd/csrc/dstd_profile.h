// dstd_profile.h -- RAII bracket of one kernel launch for the opt-in timer.
#pragma once
#include <hip/hip_runtime.h>

namespace dstd {

class ProfScope {
  public:
    ProfScope(const char *name, hipStream_t st);
    ~ProfScope();
    ProfScope(const ProfScope &) = delete;
    ProfScope &operator=(const ProfScope &) = delete;

  private:
    const char *name_;
    hipStream_t st_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
};

}  // namespace dstd
