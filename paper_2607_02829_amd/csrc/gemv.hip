// Matrix-vector products of the adaLN conditioning path (the block's modulation
// mod_b = c_b W_ada^T + b_ada and, in the backward, dc_b = dmod_b W_ada): few rows B against a
// 6D x D weight, so they are bound by reading the weight once.  Every sum runs in a fixed
// order (per lane, then a fixed butterfly or a fixed row order), so results are deterministic.
#include "common.h"
#include "sr_internal.h"

namespace sr {

constexpr int kGemvB = 8;        // rows of x handled per pass over the weight
constexpr int kGemvRows = 24;    // weight rows per chunk of the column product

template <typename T> struct Vec16T;
template <> struct Vec16T<float> { typedef float type __attribute__((ext_vector_type(4))); };
template <> struct Vec16T<bf16_t> { typedef unsigned short type __attribute__((ext_vector_type(8))); };

// Elements of one 16-byte chunk as fp32.
template <typename T>
SR_DEV void chunk_f32(i32x4 c, float (&f)[16 / sizeof(T)]) {
  typedef typename Vec16T<T>::type VT;
  const VT v = __builtin_bit_cast(VT, c);
#pragma unroll
  for (int e = 0; e < (int)(16 / sizeof(T)); ++e) f[e] = to_f32<T>((T)v[e]);
}

// One wave per output row j: lanes stride over the 16-byte chunks of W's row j.
template <typename T>
__global__ __launch_bounds__(256) void gemv_rows_kernel(const T* __restrict__ x, int ldx, const T* __restrict__ W,
                                                        const T* __restrict__ bias, int B, int J, int Dd,
                                                        float* __restrict__ y, int ldy) {
  constexpr int V = 16 / sizeof(T);
  const int lane = threadIdx.x & 63;
  const int j = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (j >= J) return;
  const int chunks = Dd / V;
  const i32x4* wr = reinterpret_cast<const i32x4*>(W + (size_t)j * Dd);
  const float bj = bias ? to_f32<T>(bias[j]) : 0.f;
  for (int b0 = 0; b0 < B; b0 += kGemvB) {
    const int nb = min(kGemvB, B - b0);
    float acc[kGemvB];
#pragma unroll
    for (int i = 0; i < kGemvB; ++i) acc[i] = 0.f;
    for (int c = lane; c < chunks; c += 64) {
      float w[V];
      chunk_f32<T>(wr[c], w);
#pragma unroll
      for (int i = 0; i < kGemvB; ++i) {
        if (i < nb) {
          float xv[V];
          chunk_f32<T>(reinterpret_cast<const i32x4*>(x + (size_t)(b0 + i) * ldx)[c], xv);
#pragma unroll
          for (int e = 0; e < V; ++e) acc[i] = fmaf(w[e], xv[e], acc[i]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kGemvB; ++i) {
      if (i < nb) {
        const float s = wave_sum(acc[i]);
        if (lane == 0) y[(size_t)(b0 + i) * ldy + j] = s + bj;
      }
    }
  }
}

// Column product, one wave per (512-column block, chunk of kGemvRows weight rows): lane l owns
// the V columns of one 16-byte chunk and sums its rows in order; the chunk's sums go to
// part[(r * B + b) * N + n], which a fixed-order column reduction adds up.
template <typename T>
__global__ __launch_bounds__(64) void gemv_cols_kernel(const float* __restrict__ x, int ldx, const T* __restrict__ W,
                                                       int B, int J, int N, float* __restrict__ part) {
  constexpr int V = 16 / sizeof(T);
  const int lane = threadIdx.x;
  const int n0 = (blockIdx.x * 64 + lane) * V;
  const int r = blockIdx.y;
  const int j0 = r * kGemvRows, j1 = min(J, j0 + kGemvRows);
  if (n0 >= N) return;
  for (int b0 = 0; b0 < B; b0 += kGemvB) {
    const int nb = min(kGemvB, B - b0);
    float acc[kGemvB][V];
#pragma unroll
    for (int i = 0; i < kGemvB; ++i)
#pragma unroll
      for (int e = 0; e < V; ++e) acc[i][e] = 0.f;
    for (int j = j0; j < j1; ++j) {
      float w[V];
      chunk_f32<T>(*reinterpret_cast<const i32x4*>(W + (size_t)j * N + n0), w);
#pragma unroll
      for (int i = 0; i < kGemvB; ++i) {
        if (i < nb) {
          const float xv = x[(size_t)(b0 + i) * ldx + j];
#pragma unroll
          for (int e = 0; e < V; ++e) acc[i][e] = fmaf(xv, w[e], acc[i][e]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < kGemvB; ++i) {
      if (i < nb) {
        float* o = part + ((size_t)r * B + b0 + i) * N + n0;
#pragma unroll
        for (int e = 0; e < V; e += 4)
          *reinterpret_cast<f32x4*>(o + e) = f32x4{acc[i][e], acc[i][e + 1], acc[i][e + 2], acc[i][e + 3]};
      }
    }
  }
}

hipError_t launch_gemv_rows(int dtype, const void* x, int ldx, const void* W, const void* bias, int B, int J, int Dd,
                            float* y, int ldy, hipStream_t st) {
  const int V = dtype == kBF16 ? 8 : 4;
  if (Dd % V != 0) return hipErrorInvalidValue;
  const dim3 g((J + 3) / 4);
  if (dtype == kBF16)
    SR_LAUNCH(gemv_rows_kernel<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)x, ldx, (const bf16_t*)W,
                       (const bf16_t*)bias, B, J, Dd, y, ldy);
  else
    SR_LAUNCH(gemv_rows_kernel<float>, g, dim3(256), 0, st, (const float*)x, ldx, (const float*)W,
                       (const float*)bias, B, J, Dd, y, ldy);
  return hipGetLastError();
}

size_t gemv_cols_scratch(int B, int J, int N) {
  return (size_t)((J + kGemvRows - 1) / kGemvRows) * B * N;
}

hipError_t launch_gemv_cols(int dtype, const float* x, int ldx, const void* W, int B, int J, int N, float* y,
                            int accumulate, float* part, hipStream_t st) {
  const int V = dtype == kBF16 ? 8 : 4;
  if (N % V != 0) return hipErrorInvalidValue;
  const int R = (J + kGemvRows - 1) / kGemvRows;
  const dim3 g((N / V + 63) / 64, R);
  if (dtype == kBF16)
    SR_LAUNCH(gemv_cols_kernel<bf16_t>, g, dim3(64), 0, st, x, ldx, (const bf16_t*)W, B, J, N, part);
  else
    SR_LAUNCH(gemv_cols_kernel<float>, g, dim3(64), 0, st, x, ldx, (const float*)W, B, J, N, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // y[b][n] (+)= sum_r part[r][b][n]: the B*N outputs as one row of width B*N (y contiguous)
  return launch_reduce_cols(part, R, 1, 1, B * N, B * N, y, nullptr, 0, st, accumulate);
}

}  // namespace sr
