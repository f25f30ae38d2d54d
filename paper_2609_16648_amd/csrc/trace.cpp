// Kernel timing with HIP events (gm_trace_*): while tracing is on, each
// launch whose kernel name matches the filter (or every n-th of them, after
// gm_trace_every(n)) is bracketed by two events on its stream; stopping waits
// for them and sums the durations per name.
#include <mutex>
#include <string>
#include <vector>

#include "../../include/gm.h"
#include "forward.h"
#include "launch.h"

namespace gm {
namespace {
struct Rec {
  const char *name;
  hipEvent_t a, b;
};
struct Sum {
  std::string name;
  int launches;
  double ms;
};
std::mutex g_mu;
bool g_on = false;
bool g_filtered = false;
int g_every = 1;       // bracket every g_every-th matching launch
long g_matched = 0;    // matching launches since gm_trace_start
std::string g_filter;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;
std::vector<Sum> g_sums;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  // timestamps only: no system-scope fence on record, whose cache write-back would leave the
  // stream idle for several microseconds on each side of a traced launch
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

TraceScope::TraceScope(const char *name, hipStream_t s) : slot(-1), stream(s) {
  if (!g_on) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on || (g_filtered && g_filter != name)) return;
  if (g_matched++ % g_every != 0) return;
  Rec r{name, take_event(), take_event()};
  if (!r.a || !r.b) return;
  (void)hipEventRecord(r.a, s);
  slot = (int)g_recs.size();
  g_recs.push_back(r);
}

TraceScope::~TraceScope() {
  if (slot < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  (void)hipEventRecord(g_recs[slot].b, stream);
}

}  // namespace gm

using namespace gm;

extern "C" gm_status gm_trace_start(const char *filter) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (auto &r : g_recs) { g_pool.push_back(r.a); g_pool.push_back(r.b); }
  g_recs.clear();
  g_sums.clear();
  g_filtered = filter != nullptr;
  g_filter = filter ? filter : "";
  g_matched = 0;
  g_on = true;
  return GM_OK;
}

extern "C" gm_status gm_trace_every(int n) {
  if (n < 1) return set_error(GM_ERR_INVALID_ARG, "gm_trace_every: n must be >= 1");
  std::lock_guard<std::mutex> lk(g_mu);
  g_every = n;
  return GM_OK;
}

extern "C" gm_status gm_trace_stop(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on = false;
  gm_status st = GM_OK;
  for (auto &r : g_recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) {
      st = GM_ERR_DEVICE;
      continue;
    }
    bool found = false;
    for (auto &s : g_sums)
      if (s.name == r.name) { s.launches += 1; s.ms += ms; found = true; break; }
    if (!found) g_sums.push_back(Sum{r.name, 1, (double)ms});
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  return st;
}

extern "C" int gm_trace_count(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  return (int)g_sums.size();
}

extern "C" gm_status gm_trace_get(int i, const char **name, int *launches, double *total_ms) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (i < 0 || i >= (int)g_sums.size()) return GM_ERR_INVALID_ARG;
  if (name) *name = g_sums[i].name.c_str();
  if (launches) *launches = g_sums[i].launches;
  if (total_ms) *total_ms = g_sums[i].ms;
  return GM_OK;
}
