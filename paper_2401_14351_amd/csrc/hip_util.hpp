// HIP runtime helpers of the loader library.
#pragma once

#include <hip/hip_runtime_api.h>

#include "common.hpp"

namespace sllm {

// Run a HIP call; on failure record the call and the HIP message and return SLLM_E_HIP.
#define SLLM_HIP(call)                                                                      \
    do {                                                                                    \
        hipError_t _e = (call);                                                             \
        if (_e != hipSuccess)                                                               \
            return ::sllm::fail(SLLM_E_HIP, "%s failed: %s", #call, hipGetErrorString(_e)); \
    } while (0)

// Make `device` current for the scope and restore the caller's device after.
class DeviceGuard {
  public:
    explicit DeviceGuard(int device) {
        if (hipGetDevice(&prev_) != hipSuccess) prev_ = -1;
        ok_ = (prev_ == device) || hipSetDevice(device) == hipSuccess;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev_ >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev_) (void)hipSetDevice(prev_);
    }
    bool ok() const { return ok_; }

  private:
    int prev_ = -1;
    bool ok_ = false;
};

}  // namespace sllm
