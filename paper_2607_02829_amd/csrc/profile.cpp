// Event-based launch timing (see profile.h) and its C entry points.
#include "profile.h"

#include "common.h"

#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/sr.h"

namespace sr {
namespace {

struct Rec {
  std::string name;
  hipEvent_t a, b;
  double flops, bytes;
};

std::mutex g_mu;
bool g_on = false;
std::string g_filter;
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

}  // namespace

LaunchHook& launch_hook() {
  static thread_local LaunchHook h;
  return h;
}

bool profiling() { return g_on; }
bool profiling_all() {
  std::lock_guard<std::mutex> lk(g_mu);
  return g_on && g_filter.empty();
}

ProfScope::ProfScope(const char* name, double flops, double bytes, hipStream_t st) : st_(st) {
  if (!g_on) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_filter.empty() && std::strstr(name, g_filter.c_str()) == nullptr) return;
  Rec r{name, take_event(), take_event(), flops, bytes};
  if (!r.a || !r.b) return;
  LaunchHook& h = launch_hook();
  if (h.start) {   // an enclosing scope that has launched nothing yet starts here
    hipEventRecord(h.start, st);
    h.start = nullptr;
  }
  outer_start_ = h.start;
  outer_stop_ = h.stop;
  launches0_ = h.launches;
  h.start = r.a;
  h.stop = r.b;
  g_recs.push_back(r);
  slot_ = (int)g_recs.size() - 1;
}

ProfScope::~ProfScope() {
  if (slot_ < 0) return;
  LaunchHook& h = launch_hook();
  std::lock_guard<std::mutex> lk(g_mu);
  if (h.launches == launches0_ && slot_ < (int)g_recs.size()) {   // nothing launched: an empty interval
    hipEventRecord(g_recs[slot_].a, st_);
    hipEventRecord(g_recs[slot_].b, st_);
  }
  h.start = outer_start_;
  h.stop = outer_stop_;
}

}  // namespace sr

extern "C" {

sr_status sr_profile_start(const char* name_filter) {
  std::lock_guard<std::mutex> lk(sr::g_mu);
  sr::g_filter = name_filter ? name_filter : "";
  sr::g_on = true;
  return SR_OK;
}

sr_status sr_profile_stop(char* out, size_t out_bytes, size_t* needed) {
  std::map<std::string, std::vector<double>> agg;   // name -> count, ms, flops, bytes
  {
    std::lock_guard<std::mutex> lk(sr::g_mu);
    sr::g_on = false;
    for (auto& r : sr::g_recs) {
      if (hipEventSynchronize(r.b) != hipSuccess) continue;
      float ms = 0.f;
      hipEventElapsedTime(&ms, r.a, r.b);
      auto& v = agg[r.name];
      if (v.empty()) v.assign(4, 0.0);
      v[0] += 1; v[1] += ms; v[2] += r.flops; v[3] += r.bytes;
      sr::g_pool.push_back(r.a);
      sr::g_pool.push_back(r.b);
    }
    sr::g_recs.clear();
  }
  std::string s;
  char line[256];
  for (auto& kv : agg) {
    snprintf(line, sizeof line, "%s %.0f %.6f %.6e %.6e\n", kv.first.c_str(), kv.second[0], kv.second[1],
             kv.second[2], kv.second[3]);
    s += line;
  }
  if (needed) *needed = s.size() + 1;
  if (out && out_bytes) {
    size_t n = std::min(out_bytes - 1, s.size());
    std::memcpy(out, s.data(), n);
    out[n] = 0;
  }
  return SR_OK;
}

}  // extern "C"
