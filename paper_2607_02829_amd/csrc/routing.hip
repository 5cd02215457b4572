// Gather and residual-delta scatter (Sec. 3.2 "Residual delta formulation",
// Eq. scatter).  Both are HBM-bound row copies: one wave per routed row, 16-byte
// vector accesses, rows of D * sizeof(T) bytes (a multiple of 16 bytes).
#include "common.h"
#include "sr_internal.h"

namespace sr {

constexpr int kRowsPerBlock = 4;   // one wave per row, 4 waves per workgroup

// h0[b,k,:] = x[b, idx[b,k], :]: two rows per wave, each pass issuing all of its loads (two
// 16-byte chunks per lane and row) before its stores.  Non-temporal accesses: a gathered row is
// read once and the copy is not re-read by this kernel, and keeping both out of the caches'
// replacement measured 0.59 -> 0.77 of 8 TB/s at 262144 rows of 2 KB.
constexpr int kGatherRows = 2;   // rows per wave

__global__ __launch_bounds__(256) void gather_kernel(const i32x4* __restrict__ x,
                                                     const int32_t* __restrict__ idx,
                                                     i32x4* __restrict__ h0, int B, int L, int K,
                                                     int chunks, int shared) {
  const int lane = threadIdx.x & 63;
  const int r0 = (blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6)) * kGatherRows;
  if (r0 >= B * K) return;
  const i32x4* src[kGatherRows];
  i32x4* dst[kGatherRows];
  bool ok[kGatherRows];
#pragma unroll
  for (int q = 0; q < kGatherRows; ++q) {
    const int r = r0 + q;
    ok[q] = r < B * K;
    const int b = ok[q] ? r / K : 0, k = ok[q] ? r - b * K : 0;
    const int i = ok[q] ? idx[(shared ? 0 : b) * K + k] : 0;
    src[q] = x + ((size_t)b * L + i) * chunks;
    dst[q] = h0 + (size_t)r * chunks;
  }
  for (int c0 = 0; c0 < chunks; c0 += 128) {
    i32x4 v[kGatherRows][2];
#pragma unroll
    for (int q = 0; q < kGatherRows; ++q)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = c0 + 64 * u + lane;
        if (ok[q] && c < chunks) v[q][u] = __builtin_nontemporal_load(src[q] + c);
      }
#pragma unroll
    for (int q = 0; q < kGatherRows; ++q)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = c0 + 64 * u + lane;
        if (ok[q] && c < chunks) __builtin_nontemporal_store(v[q][u], dst[q] + c);
      }
  }
}

// x[b,i,:] = rnd(f32(x[b,i,:]) + (f32(h[b,k,:]) - f32(h0[b,k,:]))), i = idx[b,k]
template <typename T>
__global__ __launch_bounds__(256) void scatter_delta_kernel(i32x4* __restrict__ x,
                                                            const i32x4* __restrict__ h,
                                                            const i32x4* __restrict__ h0,
                                                            const int32_t* __restrict__ idx, int B,
                                                            int L, int K, int chunks, int shared) {
#pragma clang fp contract(off)
  constexpr int V = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= B * K) return;
  const int b = r / K, k = r - b * K;
  const int i = idx[(shared ? 0 : b) * K + k];
  i32x4* xr = x + ((size_t)b * L + i) * chunks;
  const i32x4* hr = h + (size_t)r * chunks;
  const i32x4* h0r = h0 ? h0 + (size_t)r * chunks : xr;
  for (int c = lane; c < chunks; c += 64) {
    i32x4 vx = xr[c];
    i32x4 vh = __builtin_nontemporal_load(&hr[c]);
    i32x4 v0 = h0 ? __builtin_nontemporal_load(&h0r[c]) : vx;
    const T* ex = reinterpret_cast<const T*>(&vx);
    const T* eh = reinterpret_cast<const T*>(&vh);
    const T* e0 = reinterpret_cast<const T*>(&v0);
    i32x4 out;
    T* eo = reinterpret_cast<T*>(&out);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      float d = __fsub_rn(to_f32<T>(eh[e]), to_f32<T>(e0[e]));
      eo[e] = from_f32<T>(__fadd_rn(to_f32<T>(ex[e]), d));
    }
    xr[c] = out;
  }
}

// Fused forms for the stack's boundaries (one wave per routed row, 16-byte chunks of x):
// y32[b,k,:] = f32(x[b, idx[b,k], :]) (and ycopy[b,k,:] = x[b, idx[b,k], :] if given) -- the
// gather fused with the conversion of the stack's input to its fp32 residual stream;
template <typename T>
__global__ __launch_bounds__(256) void gather_rows_f32_kernel(const i32x4* __restrict__ x,
                                                              const int32_t* __restrict__ idx,
                                                              float* __restrict__ y32, i32x4* __restrict__ ycopy,
                                                              int B, int L, int K, int chunks, int shared) {
  constexpr int V = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= B * K) return;
  const int b = r / K, k = r - b * K;
  const int i = idx[(shared ? 0 : b) * K + k];
  const i32x4* xr = x + ((size_t)b * L + i) * chunks;
  float* yr = y32 + (size_t)r * chunks * V;
  for (int c = lane; c < chunks; c += 64) {
    const i32x4 v = xr[c];
    if (ycopy) ycopy[(size_t)r * chunks + c] = v;
    const T* ev = reinterpret_cast<const T*>(&v);
#pragma unroll
    for (int q = 0; q < V; q += 4) {
      f32x4 f;
#pragma unroll
      for (int e = 0; e < 4; ++e) f[e] = to_f32<T>(ev[q + e]);
      *reinterpret_cast<f32x4*>(yr + (size_t)c * V + q) = f;
    }
  }
}

// x[b,i,:] = rnd(f32(x[b,i,:]) + (f32(rnd(h32[b,k,:])) - f32(x[b,i,:]))), i = idx[b,k]: the
// residual-delta scatter with h0 re-read from x, fused with the rounding of the stack's fp32
// output to the storage type (the same values as converting h32 and then scattering).
template <typename T>
__global__ __launch_bounds__(256) void scatter_f32_delta_kernel(i32x4* __restrict__ x, const float* __restrict__ h32,
                                                                const int32_t* __restrict__ idx, int B, int L, int K,
                                                                int chunks, int shared) {
#pragma clang fp contract(off)
  constexpr int V = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
  if (r >= B * K) return;
  const int b = r / K, k = r - b * K;
  const int i = idx[(shared ? 0 : b) * K + k];
  i32x4* xr = x + ((size_t)b * L + i) * chunks;
  const float* hr = h32 + (size_t)r * chunks * V;
  for (int c = lane; c < chunks; c += 64) {
    const i32x4 vx = xr[c];
    float hv[V];
#pragma unroll
    for (int q = 0; q < V; q += 4) {
      const f32x4 f = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(hr + (size_t)c * V + q));
#pragma unroll
      for (int e = 0; e < 4; ++e) hv[q + e] = f[e];
    }
    const T* ex = reinterpret_cast<const T*>(&vx);
    i32x4 out;
    T* eo = reinterpret_cast<T*>(&out);
#pragma unroll
    for (int e = 0; e < V; ++e) {
      const float x0 = to_f32<T>(ex[e]);
      const float d = __fsub_rn(to_f32<T>(from_f32<T>(hv[e])), x0);
      eo[e] = from_f32<T>(__fadd_rn(x0, d));
    }
    xr[c] = out;
  }
}

hipError_t launch_gather_rows_f32(int dtype, int B, int L, int K, int D, const void* x, const int32_t* idx,
                                  float* y32, void* ycopy, int shared, hipStream_t st) {
  const int elt = dtype == kBF16 ? 2 : 4;
  const int chunks = D * elt / 16;
  dim3 g((B * K + kRowsPerBlock - 1) / kRowsPerBlock);
  if (dtype == kBF16)
    SR_LAUNCH(gather_rows_f32_kernel<bf16_t>, g, dim3(256), 0, st, (const i32x4*)x, idx, y32, (i32x4*)ycopy,
                       B, L, K, chunks, shared);
  else
    SR_LAUNCH(gather_rows_f32_kernel<float>, g, dim3(256), 0, st, (const i32x4*)x, idx, y32, (i32x4*)ycopy,
                       B, L, K, chunks, shared);
  return hipGetLastError();
}

hipError_t launch_scatter_f32_delta(int dtype, int B, int L, int K, int D, void* x, const float* h32,
                                    const int32_t* idx, int shared, hipStream_t st) {
  const int elt = dtype == kBF16 ? 2 : 4;
  const int chunks = D * elt / 16;
  dim3 g((B * K + kRowsPerBlock - 1) / kRowsPerBlock);
  if (dtype == kBF16)
    SR_LAUNCH(scatter_f32_delta_kernel<bf16_t>, g, dim3(256), 0, st, (i32x4*)x, h32, idx, B, L, K, chunks,
                       shared);
  else
    SR_LAUNCH(scatter_f32_delta_kernel<float>, g, dim3(256), 0, st, (i32x4*)x, h32, idx, B, L, K, chunks,
                       shared);
  return hipGetLastError();
}

hipError_t launch_gather(int elt, int B, int L, int K, int D, const void* x, const int32_t* idx, void* h0,
                         int shared, hipStream_t st) {
  const int chunks = D * elt / 16;
  constexpr int rows = kRowsPerBlock * kGatherRows;
  dim3 g((B * K + rows - 1) / rows);
  SR_LAUNCH(gather_kernel, g, dim3(256), 0, st, (const i32x4*)x, idx, (i32x4*)h0, B, L, K, chunks,
                     shared);
  return hipGetLastError();
}

hipError_t launch_scatter_delta(int dtype, int B, int L, int K, int D, void* x, const void* h, const void* h0,
                                const int32_t* idx, int shared, hipStream_t st) {
  const int elt = dtype == kBF16 ? 2 : 4;
  const int chunks = D * elt / 16;
  dim3 g((B * K + kRowsPerBlock - 1) / kRowsPerBlock);
  if (dtype == kBF16)
    SR_LAUNCH(scatter_delta_kernel<bf16_t>, g, dim3(256), 0, st, (i32x4*)x, (const i32x4*)h,
                       (const i32x4*)h0, idx, B, L, K, chunks, shared);
  else
    SR_LAUNCH(scatter_delta_kernel<float>, g, dim3(256), 0, st, (i32x4*)x, (const i32x4*)h,
                       (const i32x4*)h0, idx, B, L, K, chunks, shared);
  return hipGetLastError();
}

}  // namespace sr
