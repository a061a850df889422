// Optional kernel timing.  While tracing is on, every kernel the library
// launches is bracketed by a start/stop event pair from a preallocated pool,
// recorded on the launch stream.  Off by default; process-global; not
// thread-safe (meant for benchmarks and profiling runs).
#include <hip/hip_runtime.h>

#include <vector>

#include "../../include/treegraft.h"
#include "tg_kernels.h"

namespace tg {

namespace {
struct TraceState {
  bool on = false;
  int n = 0;
  std::vector<hipEvent_t> start, stop;
  std::vector<const char *> names;
};
TraceState g_trace;
}  // namespace

bool trace_slot(const char *name, hipEvent_t *start, hipEvent_t *stop) {
  if (!g_trace.on || g_trace.n >= (int)g_trace.start.size()) return false;
  *start = g_trace.start[g_trace.n];
  *stop = g_trace.stop[g_trace.n];
  g_trace.names[g_trace.n] = name;
  ++g_trace.n;
  return true;
}

}  // namespace tg

extern "C" {

tg_status tg_trace_begin(int capacity) {
  if (capacity <= 0 || tg::g_trace.on) return TG_ERR_INVALID_ARG;
  auto &t = tg::g_trace;
  t.start.assign(capacity, nullptr);
  t.stop.assign(capacity, nullptr);
  t.names.assign(capacity, nullptr);
  for (int i = 0; i < capacity; ++i) {
    if (hipEventCreate(&t.start[i]) != hipSuccess || hipEventCreate(&t.stop[i]) != hipSuccess)
      return TG_ERR_HIP;
  }
  t.n = 0;
  t.on = true;
  return TG_OK;
}

static tg_status trace_collect(tg_trace_record *out, int max_records, int *n_records) {
  auto &t = tg::g_trace;
  tg_status st = TG_OK;
  int n = 0;
  for (int i = 0; i < t.n; ++i) {
    float ms = 0.0f;
    if (hipEventSynchronize(t.stop[i]) != hipSuccess ||
        hipEventElapsedTime(&ms, t.start[i], t.stop[i]) != hipSuccess) {
      st = TG_ERR_HIP;
      ms = -1.0f;
    }
    if (out && n < max_records) {
      out[n].kernel = t.names[i];
      out[n].ms = ms;
      ++n;
    }
  }
  if (n_records) *n_records = n;
  return st;
}

tg_status tg_trace_read(tg_trace_record *out, int max_records, int *n_records) {
  if (!tg::g_trace.on) return TG_ERR_INVALID_ARG;
  return trace_collect(out, max_records, n_records);
}

tg_status tg_trace_end(tg_trace_record *out, int max_records, int *n_records) {
  auto &t = tg::g_trace;
  if (!t.on) return TG_ERR_INVALID_ARG;
  t.on = false;
  const tg_status st = trace_collect(out, max_records, n_records);
  for (size_t i = 0; i < t.start.size(); ++i) {
    if (t.start[i]) (void)hipEventDestroy(t.start[i]);
    if (t.stop[i]) (void)hipEventDestroy(t.stop[i]);
  }
  t.start.clear();
  t.stop.clear();
  t.names.clear();
  t.n = 0;
  return st;
}

}  // extern "C"
