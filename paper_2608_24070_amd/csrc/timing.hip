// timing.hip - optional per-kernel timing with HIP events (host code only).
// When enabled, each kernel launched by the library records a start and a stop event as part of
// its own dispatch (hipExtLaunchKernel); slim_timing_read waits for them and reports launches and
// summed milliseconds per kernel name. Off by default; costs nothing when off.
#include <hip/hip_runtime.h>

#include <algorithm>
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
struct Totals {
  long long launches = 0;
  double total_ms = 0.0;
  std::vector<float> each_ms;
};
std::map<std::string, Totals> g_total;
thread_local bool t_off = false;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  // no system-scope fence on record: it would write back L2 between the timed kernels and leave the GPU idle
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

void drain_locked() {
  for (auto& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      auto& t = g_total[p.name];
      t.launches += 1;
      t.total_ms += ms;
      t.each_ms.push_back(ms);
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
    std::vector<float> v = kv.second.each_ms;
    double med = 0.0;
    if (!v.empty()) {
      std::sort(v.begin(), v.end());
      med = v.size() % 2 ? v[v.size() / 2] : 0.5 * ((double)v[v.size() / 2 - 1] + v[v.size() / 2]);
    }
    char line[256];
    std::snprintf(line, sizeof line, "%s %lld %.6f %.6f\n", kv.first.c_str(), kv.second.launches, kv.second.total_ms, med);
    out += line;
  }
  if (!buf || buf_len == 0) return (int)out.size() + 1;
  std::snprintf(buf, buf_len, "%s", out.c_str());
  return out.size() + 1 <= buf_len ? 0 : (int)out.size() + 1;
}
