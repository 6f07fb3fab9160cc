// Per-kernel timing with HIP events (instrumentation for measurement runs).
//
// When enabled, every kernel launch of the library is bracketed by two
// events recorded on the launch stream; adept_timing_get() waits for the
// pending events and accumulates elapsed time and launch count per kernel
// name.  A name prefix can restrict the bracketing to one kernel family, so
// that a measurement run adds events (and their gaps) only around the kernel
// it measures.  Events come from a pool and are reused; nothing is allocated
// on the device.  Disabled (the default), a launch costs one relaxed atomic
// load.
#include <algorithm>
#include <atomic>
#include <cstring>
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
std::string g_prefix;   // empty: every launch is timed

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

// Resolve the oldest `n` pending pairs (blocks until they completed).
void drain(size_t n) {
  n = std::min(n, g_pending.size());
  for (size_t i = 0; i < n; ++i) {
    const Pending& p = g_pending[i];
    float ms = 0.0f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      Total& t = g_totals[p.name];
      t.launches += 1;
      t.ms += ms;
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.erase(g_pending.begin(), g_pending.begin() + n);
}

void drain() { drain(g_pending.size()); }

}  // namespace

TimedLaunch::TimedLaunch(const char* name, hipStream_t s) : name_(name), s_(s) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_prefix.empty() && strncmp(name, g_prefix.c_str(), g_prefix.size()) != 0) return;
  a_ = take_event();
  b_ = take_event();
  if (a_ && b_ && hipEventRecord((hipEvent_t)a_, s_) == hipSuccess) return;
  // no timing for this launch: the events go back to the pool
  if (a_) g_pool.push_back((hipEvent_t)a_);
  if (b_) g_pool.push_back((hipEvent_t)b_);
  a_ = b_ = nullptr;
}

TimedLaunch::~TimedLaunch() {
  if (!a_ || !b_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (hipEventRecord((hipEvent_t)b_, s_) == hipSuccess) {
    g_pending.push_back({name_, (hipEvent_t)a_, (hipEvent_t)b_});
    // the oldest half finished long ago: resolving it does not wait for
    // the queue to run dry
    if (g_pending.size() > 8192) drain(4096);
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

extern "C" adept_status adept_timing_select(const char* prefix) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_prefix = prefix ? prefix : "";
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
