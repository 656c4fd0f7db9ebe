// Kernel tracing: when enabled, every kernel launch of the library (of the
// kinds selected by the filter) is bracketed by a pair of HIP events recorded
// on the launch stream, so the caller can read per-kernel durations measured
// on the stream the kernel ran on.  The chunk launches of one aggregation
// column range share a pair (one record spanning several launches): an
// event record between back-to-back kernels costs several microseconds.  Event pairs are created once by
// pgcn_trace_enable (no allocation while tracing) without the system-scope
// fence of a default event: a fenced record writes back and invalidates the
// caches, which would slow the traced kernels themselves.  Launches beyond
// the capacity are not recorded.
#include <mutex>

#include "internal.h"

namespace pgcn {

namespace {
struct TraceState {
  std::mutex mu;
  bool on = false;
  uint32_t mask = 0xffffffffu;
  std::vector<hipEvent_t> start, stop;
  std::vector<int32_t> kind, launches;
  size_t used = 0;
};
TraceState &state() {
  static TraceState s;
  return s;
}
}  // namespace

TraceScope::TraceScope(int32_t kind, hipStream_t s) : s_(s) {
  TraceState &t = state();
  if (!t.on) return;
  std::lock_guard<std::mutex> g(t.mu);
  if (!t.on || t.used >= t.start.size() || kind < 0 || kind > 31 || !((t.mask >> kind) & 1u)) return;
  slot_ = (int64_t)t.used++;
  t.kind[slot_] = kind;
  t.launches[slot_] = 1;
  (void)hipEventRecord(t.start[slot_], s_);
}

void TraceScope::set_launches(int32_t n) {
  if (slot_ >= 0) state().launches[slot_] = n;
}

TraceScope::~TraceScope() {
  if (slot_ < 0) return;
  TraceState &t = state();
  (void)hipEventRecord(t.stop[slot_], s_);
}

}  // namespace pgcn

using namespace pgcn;

extern "C" int pgcn_trace_enable(int32_t capacity) try {
  PGCN_REQUIRE(capacity > 0 && capacity <= (1 << 20), "pgcn_trace_enable: capacity out of range");
  TraceState &t = state();
  std::lock_guard<std::mutex> g(t.mu);
  for (auto e : t.start) (void)hipEventDestroy(e);
  for (auto e : t.stop) (void)hipEventDestroy(e);
  t.start.assign(capacity, nullptr);
  t.stop.assign(capacity, nullptr);
  t.kind.assign(capacity, -1);
  t.launches.assign(capacity, 0);
  for (int32_t i = 0; i < capacity; ++i) {
    PGCN_HIP(hipEventCreateWithFlags(&t.start[i], hipEventDisableSystemFence));
    PGCN_HIP(hipEventCreateWithFlags(&t.stop[i], hipEventDisableSystemFence));
  }
  t.used = 0;
  t.mask = 0xffffffffu;
  t.on = true;
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_trace_enable");
}

extern "C" int pgcn_trace_filter(uint32_t kind_mask) try {
  TraceState &t = state();
  std::lock_guard<std::mutex> g(t.mu);
  t.mask = kind_mask;
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_trace_filter");
}

extern "C" int pgcn_trace_collect(int32_t *kinds, float *ms, int32_t *launches, int32_t max_records,
                                  int32_t *count) try {
  PGCN_REQUIRE(count && max_records >= 0 && (max_records == 0 || (kinds && ms)), "pgcn_trace_collect: bad arguments");
  TraceState &t = state();
  std::lock_guard<std::mutex> g(t.mu);
  const int32_t n = (int32_t)(t.used < (size_t)max_records ? t.used : (size_t)max_records);
  for (int32_t i = 0; i < n; ++i) {
    PGCN_HIP(hipEventSynchronize(t.stop[i]));
    float v = 0.f;
    PGCN_HIP(hipEventElapsedTime(&v, t.start[i], t.stop[i]));
    kinds[i] = t.kind[i];
    ms[i] = v;
    if (launches) launches[i] = t.launches[i];
  }
  *count = n;
  t.used = 0;
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_trace_collect");
}

extern "C" int pgcn_trace_disable(void) try {
  TraceState &t = state();
  std::lock_guard<std::mutex> g(t.mu);
  t.on = false;
  t.used = 0;
  return PGCN_OK;
} catch (...) {
  return exception_status("pgcn_trace_disable");
}
