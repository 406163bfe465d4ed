// timing.hip - optional per-kernel timing with HIP events (host code only).
// When enabled, each kernel launched by the library records a start and a stop event as part of
// its own dispatch (hipExtLaunchKernel); slim_timing_read waits for them and reports launches and
// summed milliseconds per kernel name. Off by default; costs nothing when off.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "slim_timing.h"

namespace {
struct Pending {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_mu;
bool g_on = false;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, std::pair<long long, double>> g_total;
thread_local bool t_off = false;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void drain_locked() {
  for (auto& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      auto& t = g_total[p.name];
      t.first += 1;
      t.second += ms;
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.clear();
}
}  // namespace

SlimTimingOff::SlimTimingOff() : prev(t_off) { t_off = true; }
SlimTimingOff::~SlimTimingOff() { t_off = prev; }

SlimKernelTimer::SlimKernelTimer(const char* name, hipStream_t s) : name_(name) {
  if (t_off) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on) return;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return;  // never inside a graph
  hipEvent_t a = take_event(), b = take_event();
  if (a && b) {
    a_ = a;
    b_ = b;
  } else {
    if (a) g_pool.push_back(a);
    if (b) g_pool.push_back(b);
  }
}

SlimKernelTimer::~SlimKernelTimer() {
  if (!a_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  g_pending.push_back({name_, (hipEvent_t)a_, (hipEvent_t)b_});
  if (g_pending.size() > 4096) drain_locked();
}

extern "C" int slim_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on = on != 0;
  return 0;
}

extern "C" int slim_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  drain_locked();
  g_total.clear();
  return 0;
}

extern "C" int slim_timing_read(char* buf, size_t buf_len) {
  std::lock_guard<std::mutex> lk(g_mu);
  drain_locked();
  std::string out;
  for (auto& kv : g_total) {
    char line[256];
    std::snprintf(line, sizeof line, "%s %lld %.6f\n", kv.first.c_str(), kv.second.first, kv.second.second);
    out += line;
  }
  if (!buf || buf_len == 0) return (int)out.size() + 1;
  std::snprintf(buf, buf_len, "%s", out.c_str());
  return out.size() + 1 <= buf_len ? 0 : (int)out.size() + 1;
}
