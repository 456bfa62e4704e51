// Per-device state of the launchers: the compute-unit count and the one-time
// LDS reservation of kernels that use more than 64 KiB of dynamic LDS.  Both
// are kept per device (a process may drive several GPUs) and are safe to
// reach from several host threads at once.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>

namespace q4nx {

constexpr int kMaxDevices = 64;

// Compute units of the current device (256 on MI355X), read once per device.
inline int current_device_cus() {
  static std::atomic<int> cus[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    int v = 0;
    n = (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0) ? v : 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

// A kernel's dynamic-LDS limit above the 64 KiB default must be raised with
// hipFuncSetAttribute before its first launch on each device.  One object per
// kernel (a function-local static of the kernel's launcher); the attribute is
// set once per device, and a failure is remembered and reported on every call.
class LdsReservation {
 public:
  bool ensure(const void* kernel, int bytes) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return false;
    std::call_once(once_[dev], [&] {
      ok_[dev].store(hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes) == hipSuccess,
                     std::memory_order_release);
    });
    return ok_[dev].load(std::memory_order_acquire);
  }

 private:
  std::once_flag once_[kMaxDevices];
  std::atomic<bool> ok_[kMaxDevices] = {};
};

}  // namespace q4nx
