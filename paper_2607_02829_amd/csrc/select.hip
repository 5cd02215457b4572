// Token selection kernels (Sec. 3.2 "Random token selection"; App. A.4) and the
// deterministic top-k selector, plus the index-set validator.
//
// Random: per sample, the K tokens with the smallest counter-based SplitMix64 keys,
// in ascending token order (see include/sr.h).  One workgroup per sample computes
// the keys once into LDS (up to kSelCache tokens; beyond that they are recomputed in
// every pass) and runs a radix select, 8 bits per pass from the top, for the K-th
// smallest key.  The descent stops at the first pass whose chosen digit bin is taken
// whole (the K-th key is the largest in it): then exactly the keys whose top bits are
// <= the chosen prefix are kept.  At L = 16200, K = 4050 that is two passes.  The
// kept tokens are compacted in index order with a block-wide scan.  Keys of one
// sample are distinct (mix is a bijection), so the last pass always ends the descent.
//
// Top-k: a wave per token evaluates the fp32 score in the fixed order of the
// header (16-byte chunks round-robin over 64 lanes, xor butterfly), then one
// workgroup per sample radix-selects the K largest (ties to the lower index).
#include <mutex>

#include "common.h"
#include "sr_internal.h"

namespace sr {

static constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

SR_DEV uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

// Block-wide exclusive scan of a 0/1 flag in thread order; returns the prefix and
// writes the block total to *total.  Uses `wsum` (kSelWaves ints of LDS).
SR_DEV int block_flag_scan(bool flag, int* wsum, int* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint64_t m = __ballot(flag);
  int pre = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wid] = __popcll(m);
  __syncthreads();
  int base = 0, tot = 0;
  for (int w = 0; w < kSelWaves; ++w) {
    int c = wsum[w];
    base += (w < wid) ? c : 0;
    tot += c;
  }
  __syncthreads();
  *total = tot;
  return base + pre;
}

// One radix pass: among keys with (key & mask) == prefix, histogram the digit at
// `shift`, find the digit holding the k-th smallest (1-based) and update prefix/k.
// Returns true when k equals the count of the chosen digit's bin (every key matching
// the new prefix is <= the k-th smallest).  hist: 256 ints of LDS; sh: 3 words of LDS
// for the broadcast.
template <typename KeyFn>
SR_DEV bool radix_pass(KeyFn key_of, int L, int shift, uint64_t& prefix, uint64_t& mask,
                       int& k, int* hist, uint64_t* sh) {
  for (int t = threadIdx.x; t < 256; t += blockDim.x) hist[t] = 0;
  if (threadIdx.x == 0) { sh[0] = 0; sh[1] = 1; sh[2] = 0; }
  __syncthreads();
  for (int i = threadIdx.x; i < L; i += blockDim.x) {
    uint64_t key = key_of(i);
    if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1);
  }
  __syncthreads();
  // inclusive scan of the 256 counts by the first four waves
  int cnt = 0, incl = 0;
  if (threadIdx.x < 256) {
    cnt = hist[threadIdx.x];
    incl = cnt;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int v = __shfl_up(incl, o, 64);
      if (lane >= o) incl += v;
    }
  }
  __syncthreads();
  if (threadIdx.x < 256 && (threadIdx.x & 63) == 63) hist[256 + (threadIdx.x >> 6)] = incl;
  __syncthreads();
  if (threadIdx.x < 256) {
    int w = threadIdx.x >> 6;
    for (int j = 0; j < w; ++j) incl += hist[256 + j];
    int excl = incl - cnt;
    if (cnt > 0 && excl < k && k <= incl) {
      sh[0] = (uint64_t)threadIdx.x;
      sh[1] = (uint64_t)(k - excl);
      sh[2] = (uint64_t)cnt;
    }
  }
  __syncthreads();
  uint64_t d = sh[0];
  k = (int)sh[1];
  const bool whole = (uint64_t)k == sh[2];
  prefix |= d << shift;
  mask |= 255ull << shift;
  __syncthreads();
  return whole;
}

constexpr int kSelCache = 19968;   // keys kept in LDS (156 KB) when L <= kSelCache

__global__ __launch_bounds__(kSelThreads) void select_random_kernel(int L, int K, uint64_t seed,
                                                                     uint64_t step, int32_t* idx) {
  __shared__ uint64_t kc[kSelCache];
  __shared__ int hist[256 + 4];
  __shared__ uint64_t sh[3];
  __shared__ int wsum[kSelWaves];
  const int b = blockIdx.x;
  const uint64_t s_step = mix64(seed + (step + 1ull) * kGamma);
  const uint64_t s_b = mix64(s_step + ((uint64_t)b + 1ull) * kGamma);
  auto key_of = [&](int i) { return mix64(s_b + ((uint64_t)i + 1ull) * kGamma); };
  const bool cached = L <= kSelCache;
  if (cached) {
    for (int i = threadIdx.x; i < L; i += blockDim.x) kc[i] = key_of(i);
    __syncthreads();
  }
  auto key_at = [&](int i) { return cached ? kc[i] : key_of(i); };

  uint64_t prefix = 0, mask = 0;
  int k = K;
  for (int shift = 56; shift >= 0; shift -= 8)
    if (radix_pass(key_at, L, shift, prefix, mask, k, hist, sh)) break;
  // exactly K keys have (key & mask) <= prefix: the chosen bin is taken whole

  int32_t* out = idx + (size_t)b * K;
  int base = 0;
  for (int i0 = 0; i0 < L; i0 += blockDim.x) {
    int i = i0 + threadIdx.x;
    bool f = (i < L) && ((key_at(i) & mask) <= prefix);
    int tot;
    int pos = block_flag_scan(f, wsum, &tot);
    if (f && base + pos < K) out[base + pos] = i;
    base += tot;
  }
}

// ------------------------------------------------------------------------ top-k

// One wave per token.  V = elements per 16-byte chunk (8 for bf16, 4 for fp32).
template <typename T>
__global__ __launch_bounds__(256) void topk_score_kernel(const T* __restrict__ xt,
                                                         const T* __restrict__ xp, int rows, int D,
                                                         float* __restrict__ score) {
#pragma clang fp contract(off)
  constexpr int V = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* a = xt + (size_t)row * D;
  const T* p = xp + (size_t)row * D;
  float acc = 0.0f;
  const int nchunk = D / V;
  for (int c = lane; c < nchunk; c += 64) {
    i32x4 va = *reinterpret_cast<const i32x4*>(a + c * V);
    i32x4 vp = *reinterpret_cast<const i32x4*>(p + c * V);
    const T* ea = reinterpret_cast<const T*>(&va);
    const T* ep = reinterpret_cast<const T*>(&vp);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      float d = __fsub_rn(to_f32<T>(ea[e]), to_f32<T>(ep[e]));
      acc = __fadd_rn(acc, __fmul_rn(d, d));
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) acc = __fadd_rn(acc, __shfl_xor(acc, o, 64));
  if (lane == 0) score[row] = acc;
}

constexpr int kTopkCache = 32768;   // keys kept in LDS (128 KB) when L <= kTopkCache

// The score of token i is the fp32 sum of `parts` planes of L scores each, added in plane
// order from +0 (one plane: the score itself).
__global__ __launch_bounds__(kSelThreads) void select_topk_kernel(const float* __restrict__ score,
                                                                    int parts, int L, int K, int32_t* idx) {
  __shared__ uint32_t kc[kTopkCache];
  __shared__ int hist[256 + 4];
  __shared__ uint64_t sh[3];
  __shared__ int wsum[kSelWaves];
  const int b = blockIdx.x;
  const float* sc = score + (size_t)b * parts * L;
  // Scores are >= +0, so their bit patterns order like the values; the complement
  // turns "largest" into "smallest".
  auto key_from = [&](int i) {
    float s = 0.0f;
    int p = 0;
    for (; p + 4 <= parts; p += 4) {   // four planes' loads in flight, added in plane order
      const float a0 = sc[(size_t)p * L + i], a1 = sc[(size_t)(p + 1) * L + i];
      const float a2 = sc[(size_t)(p + 2) * L + i], a3 = sc[(size_t)(p + 3) * L + i];
      s = __fadd_rn(__fadd_rn(__fadd_rn(__fadd_rn(s, a0), a1), a2), a3);
    }
    for (; p < parts; ++p) s = __fadd_rn(s, sc[(size_t)p * L + i]);
    return ~__float_as_uint(s);
  };
  const bool cached = L <= kTopkCache;
  if (cached) {
    for (int i = threadIdx.x; i < L; i += blockDim.x) kc[i] = key_from(i);
    __syncthreads();
  }
  auto key_of = [&](int i) { return (uint64_t)(cached ? kc[i] : key_from(i)); };
  uint64_t prefix = 0, mask = 0;
  int k = K;
  for (int shift = 24; shift >= 0; shift -= 8) radix_pass(key_of, L, shift, prefix, mask, k, hist, sh);
  const uint64_t thr = prefix;
  const int need_eq = k;   // how many tokens with key == thr are kept (lowest indices)

  int32_t* out = idx + (size_t)b * K;
  int base = 0, eq_base = 0;
  for (int i0 = 0; i0 < L; i0 += blockDim.x) {
    int i = i0 + threadIdx.x;
    uint64_t key = (i < L) ? key_of(i) : ~0ull;
    bool eq = (i < L) && key == thr;
    int eq_tot;
    int eq_rank = eq_base + block_flag_scan(eq, wsum, &eq_tot);
    bool f = (i < L) && (key < thr || (eq && eq_rank < need_eq));
    int tot;
    int pos = block_flag_scan(f, wsum, &tot);
    if (f && base + pos < K) out[base + pos] = i;
    base += tot;
    eq_base += eq_tot;
  }
}

// ------------------------------------------------------------------------ validation

__global__ __launch_bounds__(1024) void validate_kernel(const int32_t* idx, int rows, int K, int L,
                                                         int32_t* ok) {
  bool good = true;
  for (int t = threadIdx.x; t < rows * K; t += blockDim.x) {
    int k = t % K;
    int v = idx[t];
    if (v < 0 || v >= L) good = false;
    if (k > 0 && idx[t - 1] >= v) good = false;
  }
  int all = __syncthreads_and(good ? 1 : 0);
  if (threadIdx.x == 0) *ok = all ? 1 : 0;
}

// ------------------------------------------------------------------------ launchers

hipError_t launch_select_random(int rows, int L, int K, uint64_t seed, uint64_t step, int32_t* idx,
                                hipStream_t st) {
  SR_LAUNCH(select_random_kernel, dim3(rows), dim3(kSelThreads), 0, st, L, K, seed, step, idx);
  return hipGetLastError();
}

// Score scratch of the allocation-free top-k selection (sr_select_indices_noalloc): one array
// per GPU, held until the process ends, shared by every call on that GPU (calls that overlap on
// one GPU race).  In host code the array's name stands for a host-side shadow, not the device
// memory: kernels receive the device address that select_static_scratch() looked up.
static __device__ __align__(256) float scratch[kSelStaticScores];

hipError_t select_static_scratch(float** out) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static float* dev_ptr[kMaxDev] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!dev_ptr[dev]) {   // once per device, with that device current
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    dev_ptr[dev] = static_cast<float*>(p);
  }
  *out = dev_ptr[dev];
  return hipSuccess;
}

hipError_t launch_select_topk(int dtype, int rows, int L, int D, int K, const void* xt, const void* xp,
                              float* score, int32_t* idx, hipStream_t st) {
  const int ntok = rows * L;
  dim3 g((ntok + 3) / 4);
  if (dtype == kBF16)
    SR_LAUNCH(topk_score_kernel<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)xt, (const bf16_t*)xp,
                       ntok, D, score);
  else
    SR_LAUNCH(topk_score_kernel<float>, g, dim3(256), 0, st, (const float*)xt, (const float*)xp,
                       ntok, D, score);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  SR_LAUNCH(select_topk_kernel, dim3(rows), dim3(kSelThreads), 0, st, score, 1, L, K, idx);
  return hipGetLastError();
}

hipError_t launch_select_topk_planes(int rows, int L, int K, int parts, const float* planes, int32_t* idx,
                                     hipStream_t st) {
  SR_LAUNCH(select_topk_kernel, dim3(rows), dim3(kSelThreads), 0, st, planes, parts, L, K, idx);
  return hipGetLastError();
}

hipError_t launch_validate(const int32_t* idx, int rows, int K, int L, int32_t* ok, hipStream_t st) {
  SR_LAUNCH(validate_kernel, dim3(1), dim3(1024), 0, st, idx, rows, K, L, ok);
  return hipGetLastError();
}

}  // namespace sr
