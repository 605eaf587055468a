// Launch tracing: hipEvents recorded on the launch's stream around selected kernel launches, pooled
// and reused, summed per kernel name when tracing stops.
#include <hip/hip_runtime.h>

#include <cstring>
#include <map>
#include <mutex>
#include <sstream>
#include <string>
#include <vector>

#include "common.h"

namespace dn {
namespace {

struct Rec {
  std::string name;
  hipEvent_t a, b;
  bool ok;  // both events recorded
};

std::mutex g_mu;
bool g_on = false;
std::vector<std::string> g_filter;
std::vector<Rec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

bool wanted(const char* name) {
  if (g_filter.empty()) return true;
  for (const std::string& f : g_filter)
    if (f == name) return true;
  return false;
}

}  // namespace

TraceScope::TraceScope(const char* name, void* stream) : idx_(-1), stream_(stream) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on || !wanted(name)) return;
  hipEvent_t a = take_event(), b = take_event();
  if (!a || !b || hipEventRecord(a, (hipStream_t)stream) != hipSuccess) {  // not traced
    if (a) g_pool.push_back(a);
    if (b) g_pool.push_back(b);
    return;
  }
  g_recs.push_back(Rec{name, a, b, true});
  idx_ = (int)g_recs.size() - 1;
}

TraceScope::~TraceScope() {
  if (idx_ < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (idx_ < (int)g_recs.size() && hipEventRecord(g_recs[idx_].b, (hipStream_t)stream_) != hipSuccess)
    g_recs[idx_].ok = false;
}

}  // namespace dn

using namespace dn;

extern "C" {

int densenet_profile_start(const char* filter) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_filter.clear();
  if (filter && *filter) {
    std::stringstream ss(filter);
    std::string item;
    while (std::getline(ss, item, ','))
      if (!item.empty()) g_filter.push_back(item);
  }
  for (Rec& r : g_recs) {
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  g_on = true;
  return DN_OK;
}

int densenet_profile_stop(dn_profile_entry* out, int32_t max_entries, int32_t* n_entries) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_on = false;
  std::map<std::string, std::pair<int, double>> acc;
  std::vector<std::string> order;
  int status = DN_OK;
  for (Rec& r : g_recs) {
    float ms = 0.f;
    if (!r.ok || hipEventSynchronize(r.b) != hipSuccess ||
        hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess)
      status = fail(DN_E_HIP, "event timing failed");
    if (!acc.count(r.name)) order.push_back(r.name);
    acc[r.name].first += 1;
    acc[r.name].second += ms;
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  if (n_entries) *n_entries = (int32_t)order.size();
  for (int i = 0; i < (int)order.size() && out && i < max_entries; ++i) {
    std::memset(out[i].name, 0, sizeof(out[i].name));
    std::strncpy(out[i].name, order[i].c_str(), sizeof(out[i].name) - 1);
    out[i].launches = acc[order[i]].first;
    out[i].total_ms = acc[order[i]].second;
  }
  return status;
}

}  // extern "C"
