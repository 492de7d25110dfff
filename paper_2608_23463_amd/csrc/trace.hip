// Event-based launch tracing (see trace.hpp) and its C entry points.
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/proxyformer.h"
#include "trace.hpp"

namespace pf {

namespace {
struct Pending {
  std::string label;
  hipEvent_t start, stop;
};
struct Agg {
  int64_t launches = 0;
  double total_ms = 0.0;
};
std::mutex g_mu;
bool g_on = false;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, Agg> g_agg;
std::vector<std::string> g_order;  // labels in first-seen order
thread_local int g_open = -1;      // index in g_pending of the open launch

hipEvent_t get_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}
}  // namespace

bool trace_on() { return g_on; }

void trace_begin(const char* label, hipStream_t stream) {
  std::lock_guard<std::mutex> lk(g_mu);
  Pending p{label, get_event(), get_event()};
  if (!p.start || !p.stop) {
    if (p.start) g_pool.push_back(p.start);
    if (p.stop) g_pool.push_back(p.stop);
    return;
  }
  if (hipEventRecord(p.start, stream) != hipSuccess) {  // not traced: events back to the pool
    g_pool.push_back(p.start);
    g_pool.push_back(p.stop);
    return;
  }
  g_pending.push_back(p);
  g_open = (int)g_pending.size() - 1;
}

void trace_end(hipStream_t stream) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (g_open < 0 || g_open >= (int)g_pending.size()) return;
  if (hipEventRecord(g_pending[g_open].stop, stream) != hipSuccess) {
    // an unrecorded stop event would never complete: drop the launch from the trace
    g_pool.push_back(g_pending[g_open].start);
    g_pool.push_back(g_pending[g_open].stop);
    g_pending.erase(g_pending.begin() + g_open);
  }
  g_open = -1;
}

}  // namespace pf

using namespace pf;

extern "C" {

int proxy_trace_enable(int on) {
  std::lock_guard<std::mutex> lk(g_mu);
  const int prev = g_on ? 1 : 0;
  g_on = on != 0;
  return prev;
}

int proxy_trace_collect(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  // Launches are folded in order; each one leaves g_pending as it is counted,
  // so after a failure the launches already counted are not counted again and
  // their events (back in the pool) are referenced by nothing pending.
  size_t done = 0;
  int status = 0;
  for (; done < g_pending.size(); ++done) {
    Pending& p = g_pending[done];
    float ms = 0.0f;
    if (hipEventSynchronize(p.stop) != hipSuccess || hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess) {
      status = PF_ERR_HIP;
      break;
    }
    if (!g_agg.count(p.label)) g_order.push_back(p.label);
    Agg& a = g_agg[p.label];
    a.launches += 1;
    a.total_ms += ms;
    g_pool.push_back(p.start);
    g_pool.push_back(p.stop);
  }
  g_pending.erase(g_pending.begin(), g_pending.begin() + done);
  return status ? status : (int)g_order.size();
}

int proxy_trace_get(int i, char* label, size_t label_cap, int64_t* launches, double* total_ms) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (i < 0 || i >= (int)g_order.size() || !label || label_cap == 0) return PF_ERR_INVALID_ARG;
  const std::string& name = g_order[i];
  std::strncpy(label, name.c_str(), label_cap - 1);
  label[label_cap - 1] = '\0';
  const Agg& a = g_agg[name];
  if (launches) *launches = a.launches;
  if (total_ms) *total_ms = a.total_ms;
  return PF_OK;
}

void proxy_trace_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (Pending& p : g_pending) {
    (void)hipEventSynchronize(p.stop);  // discarded either way
    g_pool.push_back(p.start);
    g_pool.push_back(p.stop);
  }
  g_pending.clear();
  g_agg.clear();
  g_order.clear();
}

}  // extern "C"
