// Kernel tracing for libmxfp4: HIP events recorded at the start and end of
// every kernel the library launches while tracing is on (see mx_profile_start / mx_profile_stop in mxfp4.h).

#include <atomic>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "mx_internal.h"
#include "mxfp4.h"

namespace mx {
namespace {

struct Record {
  std::string name;
  hipEvent_t start, stop;
  double work;
  bool flops;
};

std::atomic<bool> g_on{false};
std::mutex g_mutex;
std::vector<Record> g_records;
std::vector<hipEvent_t> g_spare;

hipEvent_t take_event() {
  if (!g_spare.empty()) {
    hipEvent_t e = g_spare.back();
    g_spare.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

thread_local int g_no_trace = 0;

}  // namespace

bool profiling() { return g_no_trace == 0 && g_on.load(std::memory_order_acquire); }

NoTraceScope::NoTraceScope(bool active) : active_(active) {
  if (active_) ++g_no_trace;
}
NoTraceScope::~NoTraceScope() {
  if (active_) --g_no_trace;
}

TraceScope::TraceScope(const char* name, double work, bool flops) {
  if (!profiling()) return;
  std::lock_guard<std::mutex> lock(g_mutex);
  Record r{name, take_event(), take_event(), work, flops};
  if (!r.start || !r.stop) return;
  g_records.push_back(r);
  start_ = r.start;
  stop_ = r.stop;
}

}  // namespace mx

extern "C" {

int mx_profile_start(void) {
  std::lock_guard<std::mutex> lock(mx::g_mutex);
  for (auto& r : mx::g_records) {
    mx::g_spare.push_back(r.start);
    mx::g_spare.push_back(r.stop);
  }
  mx::g_records.clear();
  mx::g_on.store(true, std::memory_order_release);
  return MX_OK;
}

int mx_profile_stop(mx_kernel_stat* stats, int capacity, int* count) {
  mx::g_on.store(false, std::memory_order_release);
  std::lock_guard<std::mutex> lock(mx::g_mutex);
  std::vector<mx_kernel_stat> agg;
  int status = MX_OK;
  for (auto& r : mx::g_records) {
    float ms = 0.0f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      status = MX_ERR_HIP;
      continue;
    }
    mx_kernel_stat* s = nullptr;
    for (auto& a : agg)
      if (r.name == a.name) s = &a;
    if (!s) {
      agg.push_back(mx_kernel_stat{});
      s = &agg.back();
      std::strncpy(s->name, r.name.c_str(), sizeof(s->name) - 1);
      s->work_is_flops = r.flops ? 1 : 0;
    }
    s->launches += 1;
    s->total_ms += ms;
    s->work += r.work;
  }
  for (auto& r : mx::g_records) {  // the session's records are consumed
    mx::g_spare.push_back(r.start);
    mx::g_spare.push_back(r.stop);
  }
  mx::g_records.clear();
  if (count) *count = (int)agg.size();
  for (int i = 0; stats && i < capacity && i < (int)agg.size(); ++i) stats[i] = agg[i];
  return status;
}

}  // extern "C"
