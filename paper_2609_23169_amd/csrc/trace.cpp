// Kernel timing for the C ABI's tracing aid (ut_trace_enable /
// ut_trace_read): with tracing on, every kernel launch of the library is
// bracketed by two HIP events recorded on its own stream, so the durations are
// those of the launch stream whatever other streams do. Events are pooled and
// reused; nothing is recorded while tracing is off.
#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "common.h"

namespace ut {
namespace {

std::atomic<bool> g_on{false};
std::mutex g_mu;
struct Record {
  char name[sizeof(((ut_kernel_time*)nullptr)->name)];
  hipEvent_t start, end;
};
std::vector<Record> g_records;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {   // under g_mu
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}

}  // namespace

TraceScope::TraceScope(hipStream_t s, const char* base, int a, int b) : stream_(s) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  if (a >= 0 && b >= 0)
    snprintf(name_, sizeof(name_), "%s<%d,%d>", base, a, b);
  else if (a >= 0)
    snprintf(name_, sizeof(name_), "%s<%d>", base, a);
  else
    snprintf(name_, sizeof(name_), "%s", base);
  std::lock_guard<std::mutex> lock(g_mu);
  start_ = take_event();
  if (start_ && hipEventRecord(start_, stream_) != hipSuccess) {
    g_pool.push_back(start_);
    start_ = nullptr;
  }
}

TraceScope::~TraceScope() {
  if (!start_) return;
  std::lock_guard<std::mutex> lock(g_mu);
  hipEvent_t end = take_event();
  if (!end || hipEventRecord(end, stream_) != hipSuccess) {
    g_pool.push_back(start_);
    if (end) g_pool.push_back(end);
    return;
  }
  Record r;
  memcpy(r.name, name_, sizeof(r.name));
  r.start = start_;
  r.end = end;
  g_records.push_back(r);
}

}  // namespace ut

using namespace ut;

extern "C" {

ut_status ut_trace_enable(int on) {
  g_on.store(on != 0);
  return UT_OK;
}

int ut_trace_read(ut_kernel_time* out, int max_entries) {
  std::lock_guard<std::mutex> lock(g_mu);
  std::vector<ut_kernel_time> agg;
  int failed = 0;
  for (const Record& r : g_records) {
    float ms = 0.f;
    const bool ok = hipEventSynchronize(r.end) == hipSuccess &&
                    hipEventElapsedTime(&ms, r.start, r.end) == hipSuccess;
    g_pool.push_back(r.start);
    g_pool.push_back(r.end);
    if (!ok) {
      ++failed;
      continue;
    }
    ut_kernel_time* k = nullptr;
    for (auto& e : agg)
      if (strcmp(e.name, r.name) == 0) k = &e;
    if (!k) {
      agg.push_back(ut_kernel_time{});
      k = &agg.back();
      memcpy(k->name, r.name, sizeof(k->name));
      k->min_ms = ms;
      k->max_ms = ms;
    }
    k->count += 1;
    k->total_ms += ms;
    if (ms < k->min_ms) k->min_ms = ms;
    if (ms > k->max_ms) k->max_ms = ms;
  }
  g_records.clear();
  if (failed) {
    fail(UT_ERR_HIP, "ut_trace_read: %d launch timings could not be read", failed);
    return -1;
  }
  const int n = (int)agg.size();
  for (int i = 0; i < n && i < max_entries && out; ++i) out[i] = agg[i];
  return n;
}

}  // extern "C"
