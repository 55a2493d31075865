// Optional per-kernel timing: when enabled, every kernel launch of the library
// is bracketed by HIP events recorded on the launch stream, so a caller can read
// the device time of each kernel without an external profiler.
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace seg {
namespace {
struct Rec {
  std::string name;
  hipEvent_t start, stop;
};
std::mutex g_mu;
std::vector<Rec> g_recs;
// read by every launch of any thread, written by seg_profile_enable
std::atomic<bool> g_on{false};

void destroy_pair(hipEvent_t a, hipEvent_t b) {
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
}
}  // namespace

ProfScope::ProfScope(const char *name, hipStream_t s) : name_(name), stream_(s) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  if (hipEventCreate(&start_) != hipSuccess) return;
  if (hipEventCreate(&stop_) != hipSuccess) {
    (void)hipEventDestroy(start_);
    return;
  }
  if (hipEventRecord(start_, stream_) != hipSuccess) {
    destroy_pair(start_, stop_);
    return;
  }
  active_ = true;
}

ProfScope::~ProfScope() {
  if (!active_) return;
  if (hipEventRecord(stop_, stream_) != hipSuccess) {
    destroy_pair(start_, stop_);
    return;
  }
  std::lock_guard<std::mutex> lk(g_mu);
  g_recs.push_back({name_, start_, stop_});
}

}  // namespace seg

using namespace seg;

extern "C" void seg_profile_enable(int32_t on) { g_on.store(on != 0, std::memory_order_relaxed); }

extern "C" void seg_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (auto &r : g_recs) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_recs.clear();
}

extern "C" seg_status seg_profile_read(const char *name, double *total_ms, int64_t *launches) {
  return guarded([&] {
    SEG_CHECK(name && total_ms && launches, SEG_ERR_ARG, "NULL argument");
    std::lock_guard<std::mutex> lk(g_mu);
    double tot = 0.0;
    int64_t n = 0;
    for (auto &r : g_recs) {
      if (r.name != name) continue;
      SEG_HIP(hipEventSynchronize(r.stop));
      float ms = 0.f;
      SEG_HIP(hipEventElapsedTime(&ms, r.start, r.stop));
      tot += ms;
      ++n;
    }
    *total_ms = tot;
    *launches = n;
  });
}
