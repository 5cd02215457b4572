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

// Sustained bf16 matrix-core rate: eight waves per CU (two per SIMD), each issuing independent
// v_mfma_f32_32x32x16_bf16 into eight accumulators, no memory traffic in the loop.  One
// workgroup per CU, so the launch is a single round.
constexpr int kProbeIters = 4096, kProbeAcc = 8;

__global__ __launch_bounds__(512) void mfma_probe_kernel(float* sink, int iters) {
  f32x16 acc[kProbeAcc];
  for (int i = 0; i < kProbeAcc; ++i)
    for (int r = 0; r < 16; ++r) acc[i][r] = 0.f;
  i32x4 a = {(int)threadIdx.x, 0x3f803f80, 0x3f003f00, (int)blockIdx.x};
  i32x4 b = {0x3c003c00, (int)threadIdx.x, 0x3e003e00, 0x3d003d00};
  asm volatile("" : "+v"(a), "+v"(b));   // opaque operands: nothing folds
  for (int it = 0; it < iters; ++it)
#pragma unroll
    for (int i = 0; i < kProbeAcc; ++i)
      acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b),
                                                       acc[i], 0, 0, 0);
  float s = 0.f;
  for (int i = 0; i < kProbeAcc; ++i)
    for (int r = 0; r < 16; ++r) s += acc[i][r];
  if (threadIdx.x == 0) sink[0] = s;   // keeps the work; every workgroup writes the same word
}

hipError_t probe_mfma_rate(float* sink, double* tflops, hipStream_t st) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  hipEvent_t a = nullptr, b = nullptr;
  if ((e = hipEventCreate(&a)) != hipSuccess) return e;
  if ((e = hipEventCreate(&b)) != hipSuccess) {
    hipEventDestroy(a);
    return e;
  }
  SR_LAUNCH(mfma_probe_kernel, dim3(cus), dim3(512), 0, st, sink, kProbeIters);   // warm-up (clock ramp)
  e = hipEventRecord(a, st);
  if (e == hipSuccess) SR_LAUNCH(mfma_probe_kernel, dim3(cus), dim3(512), 0, st, sink, kProbeIters);
  if (e == hipSuccess) e = hipGetLastError();
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  hipEventDestroy(a);
  hipEventDestroy(b);
  if (e != hipSuccess) return e;
  const double flops = (double)cus * 8 * kProbeIters * kProbeAcc * (2.0 * 32 * 32 * 16);
  *tflops = ms > 0.f ? flops / (ms * 1e-3) / 1e12 : 0.0;
  return hipSuccess;
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
