// Host-side helper shared by the C ABI implementations: make a handle's device
// current for the duration of one call and give the caller back the device it
// had, on every return path.
#pragma once

#include <hip/hip_runtime.h>

namespace kvshot {

class DeviceGuard {
 public:
  explicit DeviceGuard(int device) {
    if (hipGetDevice(&prev_) != hipSuccess) {
      ok_ = false;
      return;
    }
    if (prev_ != device) {
      ok_ = hipSetDevice(device) == hipSuccess;
      switched_ = ok_;
    }
  }
  ~DeviceGuard() {
    if (switched_) (void)hipSetDevice(prev_);
  }
  DeviceGuard(const DeviceGuard&) = delete;
  DeviceGuard& operator=(const DeviceGuard&) = delete;
  bool ok() const { return ok_; }

 private:
  int prev_ = -1;
  bool ok_ = true;
  bool switched_ = false;
};

}  // namespace kvshot
