// Optional HIP-event timing of the library's kernels, for benchmarks.  When
// enabled, each launch of a tracked kernel is bracketed by a pair of events
// recorded on the launch's own stream; duo_profile_read sums the elapsed
// times.  Meant for single-threaded benchmark drivers.
#include <hip/hip_runtime.h>

#include <mutex>
#include <utility>
#include <vector>

#include "internal.h"

namespace duo {

namespace {

struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending[DUO_PROF_COUNT];
  std::vector<hipEvent_t> pool;
  double total_ms[DUO_PROF_COUNT] = {};
  long long count[DUO_PROF_COUNT] = {};

  hipEvent_t get() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
  }
};

Profiler& prof() {
  static Profiler p;
  return p;
}

}  // namespace

void prof_begin(int id, hipStream_t s) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (!p.on) return;
  hipEvent_t a = p.get(), b = p.get();
  if (!a || !b) return;
  hipEventRecord(a, s);
  p.pending[id].push_back({a, b});
}

void prof_end(int id, hipStream_t s) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (!p.on || p.pending[id].empty()) return;
  hipEventRecord(p.pending[id].back().second, s);
}

}  // namespace duo

using namespace duo;

extern "C" {

duo_status duo_profile_enable(int32_t on) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.on = on != 0;
  return DUO_OK;
}

duo_status duo_profile_read(int32_t kernel, double* total_ms, int64_t* launches) {
  if (kernel < 0 || kernel >= DUO_PROF_COUNT || !total_ms || !launches) return DUO_ERR_INVALID_ARG;
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& pr : p.pending[kernel]) {
    if (hipEventSynchronize(pr.second) != hipSuccess) return DUO_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, pr.first, pr.second) != hipSuccess) return DUO_ERR_HIP;
    p.total_ms[kernel] += ms;
    p.count[kernel] += 1;
    p.pool.push_back(pr.first);
    p.pool.push_back(pr.second);
  }
  p.pending[kernel].clear();
  *total_ms = p.total_ms[kernel];
  *launches = p.count[kernel];
  p.total_ms[kernel] = 0.0;
  p.count[kernel] = 0;
  return DUO_OK;
}

}  // extern "C"
