// Makes a plan's device current for the length of a scope and restores the
// caller's device afterwards, for the synchronous calls (status, reset,
// trace, occupancy) that may come while another device is current.
#pragma once

#include <hip/hip_runtime.h>

namespace ebag {

class DeviceGuard {
 public:
  explicit DeviceGuard(int device) {
    if (hipGetDevice(&prev_) != hipSuccess) {
      err_ = hipErrorInvalidDevice;
      return;
    }
    if (prev_ != device) {
      err_ = hipSetDevice(device);
      switched_ = err_ == hipSuccess;
    }
  }
  ~DeviceGuard() {
    if (switched_) (void)hipSetDevice(prev_);
  }
  DeviceGuard(const DeviceGuard&) = delete;
  DeviceGuard& operator=(const DeviceGuard&) = delete;
  // hipSuccess when the plan's device is current.
  hipError_t error() const { return err_; }

 private:
  int prev_ = -1;
  bool switched_ = false;
  hipError_t err_ = hipSuccess;
};

}  // namespace ebag
