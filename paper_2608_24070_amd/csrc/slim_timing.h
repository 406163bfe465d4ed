// slim_timing.h - scoped per-kernel HIP-event timer used around each library launch.
#pragma once

#include <hip/hip_runtime.h>

class SlimKernelTimer {
 public:
  SlimKernelTimer(const char* name, hipStream_t s);
  void stop();
  ~SlimKernelTimer() { stop(); }

 private:
  const char* name_;
  hipStream_t s_;
  void* a_ = nullptr;
  void* b_ = nullptr;
  bool active_ = false;
};
