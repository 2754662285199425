// Optional HIP-event timing of the library's kernels, for benchmarks.  When
// enabled, each launch of a tracked kernel is bracketed by a pair of events
// recorded on the launch's own stream; duo_profile_read sums the elapsed
// times.  Meant for single-threaded benchmark drivers.
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "internal.h"

namespace duo {

namespace {

struct Bracket {
  hipEvent_t a, b;
  bool ended;  // the end event was recorded
};

struct Profiler {
  std::mutex mu;
  bool on = false;
  std::vector<Bracket> pending[DUO_PROF_COUNT];
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
  void put(hipEvent_t e) {
    if (e) pool.push_back(e);
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
  if (!a || !b || hipEventRecord(a, s) != hipSuccess) {  // this launch goes untimed
    p.put(a);
    p.put(b);
    return;
  }
  p.pending[id].push_back({a, b, false});
}

void prof_end(int id, hipStream_t s) {
  Profiler& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  if (!p.on || p.pending[id].empty() || p.pending[id].back().ended) return;
  Bracket& br = p.pending[id].back();
  if (hipEventRecord(br.b, s) == hipSuccess) {
    br.ended = true;
  } else {  // this launch goes untimed
    p.put(br.a);
    p.put(br.b);
    p.pending[id].pop_back();
  }
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
  duo_status st = DUO_OK;
  for (const Bracket& br : p.pending[kernel]) {
    float ms = 0.f;
    if (br.ended) {  // a bracket left open (no end recorded) is dropped
      if (hipEventSynchronize(br.b) == hipSuccess && hipEventElapsedTime(&ms, br.a, br.b) == hipSuccess) {
        p.total_ms[kernel] += ms;
        p.count[kernel] += 1;
      } else {
        st = DUO_ERR_HIP;
      }
    }
    p.put(br.a);
    p.put(br.b);
  }
  p.pending[kernel].clear();
  *total_ms = p.total_ms[kernel];
  *launches = p.count[kernel];
  p.total_ms[kernel] = 0.0;
  p.count[kernel] = 0;
  return st;
}

}  // extern "C"
