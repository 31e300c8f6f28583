// Opt-in kernel timing for benchmarks: while enabled, every kernel the
// library launches is bracketed by a pair of HIP events on the launch stream.
// Reading waits for the recorded events and aggregates durations per kernel.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "sgdkv.h"
#include "sgdkv_internal.h"

namespace sgdkv {
namespace {

struct Pending {
  const char* name;
  hipEvent_t start, stop;
};

std::atomic<bool> g_on{false};
std::mutex g_mu;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_free;
struct Total {
  int64_t count = 0;
  double ms = 0.0;
};
std::map<std::string, Total> g_totals;
thread_local Pending t_open{nullptr, nullptr, nullptr};

hipEvent_t take_event() {
  if (!g_free.empty()) {
    hipEvent_t e = g_free.back();
    g_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Waits for and folds every recorded pair into the totals (g_mu held).
void drain() {
  for (const Pending& p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.stop) == hipSuccess && hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
      Total& t = g_totals[p.name];
      t.count += 1;
      t.ms += ms;
    }
    g_free.push_back(p.start);
    g_free.push_back(p.stop);
  }
  g_pending.clear();
}

}  // namespace

void prof_begin(const char* name, hipStream_t stream) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lock(g_mu);
  t_open.name = name;
  t_open.start = take_event();
  t_open.stop = take_event();
  if (t_open.start && t_open.stop) (void)hipEventRecord(t_open.start, stream);
}

void prof_end(hipStream_t stream) {
  if (!g_on.load(std::memory_order_relaxed) || !t_open.name) return;
  std::lock_guard<std::mutex> lock(g_mu);
  if (t_open.start && t_open.stop) {
    (void)hipEventRecord(t_open.stop, stream);
    g_pending.push_back(t_open);
  }
  t_open = Pending{nullptr, nullptr, nullptr};
}

}  // namespace sgdkv

extern "C" {

sgdkv_status sgdkv_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lock(sgdkv::g_mu);
  sgdkv::g_on.store(on != 0);
  return SGDKV_OK;
}

sgdkv_status sgdkv_profile_reset(void) {
  std::lock_guard<std::mutex> lock(sgdkv::g_mu);
  sgdkv::drain();
  sgdkv::g_totals.clear();
  return SGDKV_OK;
}

sgdkv_status sgdkv_profile_read(int32_t max_entries, char* names, int64_t* counts, double* total_ms,
                                int32_t* n_out) {
  if (max_entries < 0 || !n_out || (max_entries > 0 && (!names || !counts || !total_ms)))
    return SGDKV_ERR_INVALID_ARG;
  std::lock_guard<std::mutex> lock(sgdkv::g_mu);
  sgdkv::drain();
  int32_t n = 0;
  for (const auto& kv : sgdkv::g_totals) {
    if (n < max_entries) {
      std::strncpy(names + (size_t)n * 64, kv.first.c_str(), 63);
      names[(size_t)n * 64 + 63] = '\0';
      counts[n] = kv.second.count;
      total_ms[n] = kv.second.ms;
    }
    ++n;
  }
  *n_out = n;
  return SGDKV_OK;
}

}  // extern "C"
