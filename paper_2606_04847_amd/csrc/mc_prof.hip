// Opt-in per-kernel timing.  When enabled, every internal launch is bracketed
// by a pair of hipEvents recorded on the launch stream, tagged with the
// kernel's name and its algorithmic FLOPs and bytes; mc_profiler_read waits
// for the events and folds them into per-name totals.  Disabled (the
// default), it costs one relaxed atomic load per launch.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "mc_internal.hpp"

namespace mc {

namespace {

struct Pending {
  const char* name;
  hipEvent_t start, stop;
  double flops, bytes;
};

struct Total {
  std::string name;
  int64_t launches = 0;
  double ms = 0.0, flops = 0.0, bytes = 0.0;
};

std::atomic<int> g_on{0};
std::mutex g_mu;
std::vector<Pending> g_pending;
std::vector<Total> g_totals;

void fold_locked() {
  for (Pending& p : g_pending) {
    float ms = 0.0f;
    (void)hipEventSynchronize(p.stop);
    (void)hipEventElapsedTime(&ms, p.start, p.stop);
    (void)hipEventDestroy(p.start);
    (void)hipEventDestroy(p.stop);
    Total* t = nullptr;
    for (Total& x : g_totals)
      if (x.name == p.name) t = &x;
    if (!t) {
      g_totals.push_back(Total{});
      t = &g_totals.back();
      t->name = p.name;
    }
    t->launches += 1;
    t->ms += ms;
    t->flops += p.flops;
    t->bytes += p.bytes;
  }
  g_pending.clear();
}

}  // namespace

ProfScope::ProfScope(hipStream_t s, const char* name, double flops, double bytes)
    : stream_(s), name_(name), flops_(flops), bytes_(bytes) {
  if (name_ == nullptr || !g_on.load(std::memory_order_relaxed)) return;
  if (hipEventCreate(&start_) != hipSuccess) return;
  if (hipEventCreate(&stop_) != hipSuccess) {
    (void)hipEventDestroy(start_);
    return;
  }
  (void)hipEventRecord(start_, stream_);
  active_ = true;
}

ProfScope::~ProfScope() {
  if (!active_) return;
  (void)hipEventRecord(stop_, stream_);
  std::lock_guard<std::mutex> lk(g_mu);
  g_pending.push_back(Pending{name_, start_, stop_, flops_, bytes_});
}

}  // namespace mc

extern "C" {

void mc_profiler_enable(int32_t on) { mc::g_on.store(on ? 1 : 0); }

void mc_profiler_reset(void) {
  std::lock_guard<std::mutex> lk(mc::g_mu);
  mc::fold_locked();
  mc::g_totals.clear();
}

int32_t mc_profiler_read(mc_kernel_time_t* out, int32_t cap) {
  std::lock_guard<std::mutex> lk(mc::g_mu);
  mc::fold_locked();
  const int32_t n = int32_t(mc::g_totals.size());
  for (int32_t i = 0; i < n && i < cap && out; ++i) {
    const mc::Total& t = mc::g_totals[i];
    std::memset(out[i].name, 0, sizeof(out[i].name));
    std::strncpy(out[i].name, t.name.c_str(), sizeof(out[i].name) - 1);
    out[i].launches = t.launches;
    out[i].total_ms = t.ms;
    out[i].total_flops = t.flops;
    out[i].total_bytes = t.bytes;
  }
  return n;
}

}  // extern "C"
