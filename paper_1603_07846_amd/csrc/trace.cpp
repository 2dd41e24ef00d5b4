// trace.cpp -- optional per-kernel timing: when enabled, every launch of the
// library is bracketed by two timing events recorded on the launch stream,
// tagged with the kernel's name and its algorithmic work (flops or bytes).
// Off by default; when off a launch site costs one relaxed atomic load.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <vector>

#include "internal.h"

namespace singa {

namespace {

struct Record {
  const char* name;
  hipEvent_t start, stop;
  double work;
  int unit;
};

constexpr size_t kMaxRecords = 1 << 16;

std::atomic<int> g_on{0};
std::mutex g_mu;
std::vector<Record> g_records;      // recorded since the last enable
std::vector<hipEvent_t> g_free;     // events kept for reuse

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

}  // namespace

TraceScope::TraceScope(const char* name, hipStream_t st, double work, int unit) : st_(st), idx_(-1) {
  if (!g_on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_records.size() >= kMaxRecords) return;
  Record r{name, take_event(), take_event(), work, unit};
  if (!r.start || !r.stop || hipEventRecord(r.start, st) != hipSuccess) {
    if (r.start) g_free.push_back(r.start);
    if (r.stop) g_free.push_back(r.stop);
    return;
  }
  idx_ = (long)g_records.size();
  g_records.push_back(r);
}

TraceScope::~TraceScope() {
  if (idx_ < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  // a failed record leaves this launch untimed; the trace is diagnostic only
  if ((size_t)idx_ < g_records.size()) (void)hipEventRecord(g_records[idx_].stop, st_);
}

}  // namespace singa

extern "C" {

int singa_trace_enable(int on) {
  using namespace singa;
  std::lock_guard<std::mutex> lk(g_mu);
  if (on) {
    for (auto& r : g_records) {
      g_free.push_back(r.start);
      g_free.push_back(r.stop);
    }
    g_records.clear();
  }
  g_on.store(on ? 1 : 0);
  return 0;
}

int singa_trace_count(void) {
  using namespace singa;
  std::lock_guard<std::mutex> lk(g_mu);
  return (int)g_records.size();
}

int singa_trace_get(int i, const char** name, double* ms, double* work, int* unit) {
  using namespace singa;
  if (!name || !ms || !work || !unit) return -1;
  std::lock_guard<std::mutex> lk(g_mu);
  if (i < 0 || (size_t)i >= g_records.size()) return -2;
  const Record& r = g_records[i];
  float t = 0.f;
  if (hipEventElapsedTime(&t, r.start, r.stop) != hipSuccess) return -6;
  *name = r.name;
  *ms = t;
  *work = r.work;
  *unit = r.unit;
  return 0;
}

}  // extern "C"
