// Per-kernel timing with HIP events (instrumentation for measurement runs).
//
// When enabled, every kernel launch of the library is bracketed by two
// events recorded on the launch stream; adept_timing_get() waits for the
// pending events and accumulates elapsed time and launch count per kernel
// name.  Events come from a pool and are reused; nothing is allocated on the
// device.  Disabled (the default), a launch costs one relaxed atomic load.
#include <atomic>
#include <map>
#include <mutex>
#include <vector>

#include "common.h"

namespace adept {
namespace {

struct Pending {
  const char* name;
  hipEvent_t a, b;
};
struct Total {
  int64_t launches = 0;
  double ms = 0.0;
};

std::atomic<int> g_on{0};
std::mutex g_mu;
std::vector<hipEvent_t> g_pool;
std::vector<Pending> g_pending;
std::map<std::string, Total> g_totals;

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

// Resolve all pending pairs (blocks until they completed).
void drain() {
  for (auto& p : g_pending) {
    float ms = 0.0f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      Total& t = g_totals[p.name];
      t.launches += 1;
      t.ms += ms;
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.clear();
}

}  // namespace

TimedLaunch::TimedLaunch(const char* name, hipStream_t s) : name_(name), s_(s) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  a_ = take_event();
  b_ = take_event();
  if (a_ && b_) hipEventRecord((hipEvent_t)a_, s_);
}

TimedLaunch::~TimedLaunch() {
  if (!a_ || !b_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (hipEventRecord((hipEvent_t)b_, s_) == hipSuccess) {
    g_pending.push_back({name_, (hipEvent_t)a_, (hipEvent_t)b_});
    if (g_pending.size() > 8192) drain();
  } else {
    g_pool.push_back((hipEvent_t)a_);
    g_pool.push_back((hipEvent_t)b_);
  }
}

}  // namespace adept

using namespace adept;

extern "C" adept_status adept_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on.store(on ? 1 : 0);
  return ADEPT_OK;
}

extern "C" void adept_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  drain();
  g_totals.clear();
}

extern "C" int adept_timing_count(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  drain();
  return (int)g_totals.size();
}

extern "C" adept_status adept_timing_get(int idx, char* name, int name_len, int64_t* launches,
                                         double* total_ms) {
  std::lock_guard<std::mutex> lk(g_mu);
  drain();
  ADEPT_REQUIRE(idx >= 0 && idx < (int)g_totals.size(), "timing_get: index %d out of range", idx);
  ADEPT_REQUIRE(name && name_len > 0 && launches && total_ms, "timing_get: NULL output");
  auto it = g_totals.begin();
  std::advance(it, idx);
  snprintf(name, (size_t)name_len, "%s", it->first.c_str());
  *launches = it->second.launches;
  *total_ms = it->second.ms;
  return ADEPT_OK;
}
