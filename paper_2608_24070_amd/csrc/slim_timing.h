// slim_timing.h - optional per-kernel timing of the library's launches.
// A SlimKernelTimer names one launch; when timing is on (and the stream is not being captured)
// it hands out a start and a stop event that the launch itself records through
// hipExtLaunchKernel, so they carry the kernel's own begin and end timestamps, not the time of
// separate event packets around it. SLIM_LAUNCH launches through it.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

class SlimKernelTimer {
 public:
  SlimKernelTimer(const char* name, hipStream_t s);
  ~SlimKernelTimer();
  hipEvent_t start() const { return (hipEvent_t)a_; }
  hipEvent_t stop() const { return (hipEvent_t)b_; }

 private:
  const char* name_;
  void* a_ = nullptr;
  void* b_ = nullptr;
};

// While one of these lives on a thread, the library's launches on that thread record no events.
struct SlimTimingOff {
  SlimTimingOff();
  ~SlimTimingOff();
  bool prev;
};

// untimed launches (timing off, or a stream under graph capture) take the plain launch path
#define SLIM_LAUNCH(timer, kernel, grid, block, stream, ...)                                               \
  do {                                                                                                    \
    if ((timer).start())                                                                                  \
      hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, (timer).start(), (timer).stop(), 0, __VA_ARGS__); \
    else                                                                                                  \
      hipLaunchKernelGGL(kernel, grid, block, 0, stream, __VA_ARGS__);                                    \
  } while (0)
