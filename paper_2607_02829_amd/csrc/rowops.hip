// Row-wise and column-wise kernels of the block: LayerNorm forward/backward (with
// the optional adaLN modulation), deterministic column reductions (bias and
// modulation gradients), dtype conversion, and the attention row-sum
// delta_i = sum_d dO[i,d] * O[i,d].
//
// LayerNorm (block of Sec. 3.3): y = (x - mean) * rstd * gamma + beta, biased
// variance over D, two-pass mean/variance in fp32 registers, one wave per row.
// With adaLN the affine step is replaced by y = xhat * (1 + scale_b) + shift_b.
#include "common.h"
#include "sr_internal.h"

namespace sr {

constexpr int kMaxPerLane = 32;   // D <= 2048

// Lane-to-column map of the row kernels: with V = 4 (D % 256 == 0) lane l owns the 16-byte
// groups of columns 4l + 256j .. 4l + 256j + 3; with V = 1 it owns columns l + 64j.
template <int V> SR_DEV int col_of(int lane, int j) { return (lane + 64 * j) * V; }

template <int V> SR_DEV void ldv(const float* p, float* o) {
  if constexpr (V == 4) {
    f32x4 v = *reinterpret_cast<const f32x4*>(p);
    o[0] = v[0]; o[1] = v[1]; o[2] = v[2]; o[3] = v[3];
  } else {
    o[0] = p[0];
  }
}
template <int V> SR_DEV void ldv(const bf16_t* p, float* o) {
  if constexpr (V == 4) {
    i32x2 w = *reinterpret_cast<const i32x2*>(p);
    const bf16_t* e = reinterpret_cast<const bf16_t*>(&w);
    o[0] = bf2f(e[0]); o[1] = bf2f(e[1]); o[2] = bf2f(e[2]); o[3] = bf2f(e[3]);
  } else {
    o[0] = bf2f(p[0]);
  }
}
template <int V> SR_DEV void stv(float* p, const float* v) {
  if constexpr (V == 4) {
    f32x4 w = {v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(p) = w;
  } else {
    p[0] = v[0];
  }
}
template <int V> SR_DEV void stv(bf16_t* p, const float* v) {
  if constexpr (V == 4) {
    i32x2 w;
    w[0] = (int)f2bf2(v[0], v[1]);
    w[1] = (int)f2bf2(v[2], v[3]);
    *reinterpret_cast<i32x2*>(p) = w;
  } else {
    p[0] = f2bf(v[0]);
  }
}

// x: fp32 [M, D]; mod (adaLN): fp32 [B, 6D] with shift at mod_off, scale at mod_off + D.
// One row per wave.  NJC > 0: every lane holds exactly NJC groups of V columns (D = 64 V NJC,
// all loads unconditional and issued together); NJC = 0: any D <= 64 V kMaxPerLane.
// GATHER: the input row is token i = gidx[(gshared ? 0 : b) * S + s] of sample b of the token
// sequence gsrc [B, gL, D] (storage type), for row m = b * S + s; its fp32 values are also
// written to xcopy[m] (the residual stream the block keeps): the gather of the routed rows and
// the first LayerNorm in one pass, with the values and arithmetic of the separate steps.
// APPLY: mean and rstd are read from mean_out / rstd_out (the forward's statistics) instead of
// computed, and nothing else is written but y: the LayerNorm output recomputed bit for bit.
template <typename T, typename Ta, int V, int NJC, bool GATHER = false, bool APPLY = false>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const float* __restrict__ x, const T* __restrict__ gamma,
                                                     const T* __restrict__ beta, const float* __restrict__ mod,
                                                     int mod_off, int M, int S, int D, float eps,
                                                     Ta* __restrict__ y, float* __restrict__ mean_out,
                                                     float* __restrict__ rstd_out, const T* __restrict__ gsrc,
                                                     const int32_t* __restrict__ gidx, int gL,
                                                     int gshared, float* __restrict__ xcopy) {
  constexpr int NJ = NJC > 0 ? NJC : kMaxPerLane / V;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int n = NJC > 0 ? NJC : D / (64 * V);
  const float* xr = x + (size_t)row * D;
  const int b = row / S;
  const T* gr = nullptr;
  if constexpr (GATHER) {
    const int i = gidx[(size_t)(gshared ? 0 : b) * S + (row - b * S)];
    gr = gsrc + ((size_t)b * gL + i) * D;
  }
  const float* shift = mod ? mod + (size_t)b * 6 * D + mod_off : nullptr;
  float v[NJ][V], w[NJ][V], bb[NJ][V];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (j < n) {
      const int c = col_of<V>(lane, j);
      if constexpr (GATHER) ldv<V>(gr + c, v[j]);
      else ldv<V>(xr + c, v[j]);
      if (mod) {
        ldv<V>(shift + D + c, w[j]);
        ldv<V>(shift + c, bb[j]);
      } else {
        ldv<V>(gamma + c, w[j]);
        ldv<V>(beta + c, bb[j]);
      }
    }
  if constexpr (GATHER) {
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < n) stv<V>(xcopy + (size_t)row * D + col_of<V>(lane, j), v[j]);
  }
  float mean, rstd;
  if constexpr (APPLY) {
    mean = mean_out[row];
    rstd = rstd_out[row];
  } else {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < n)
#pragma unroll
        for (int e = 0; e < V; ++e) s += v[j][e];
    mean = wave_sum(s) / (float)D;
    float q = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if (j < n)
#pragma unroll
        for (int e = 0; e < V; ++e) { const float d = v[j][e] - mean; q += d * d; }
    rstd = 1.0f / sqrtf(wave_sum(q) / (float)D + eps);
  }
  Ta* yr = y + (size_t)row * D;
#pragma unroll
  for (int j = 0; j < NJ; ++j)
    if (j < n) {
      float o[V];
#pragma unroll
      for (int e = 0; e < V; ++e) o[e] = (v[j][e] - mean) * rstd * (mod ? w[j][e] + 1.0f : w[j][e]) + bb[j][e];
      stv<V>(yr + col_of<V>(lane, j), o);
    }
  if constexpr (!APPLY) {
    if (lane == 0) { mean_out[row] = mean; rstd_out[row] = rstd; }
  }
}

// Backward.  du: fp32 [M, D] gradient of the LayerNorm output (after modulation);
// dres: fp32 [M, D] residual gradient added to the result (may alias dx).
// dx = dres + (dxhat - mean(dxhat) - xhat * mean(dxhat * xhat)) * rstd with
// dxhat = du * gamma (or du * (1 + scale_b)).  A workgroup takes kLnBwdRows rows of one
// sample (two per wave, loads issued together) and writes partial column
// sums of du * xhat and du to part[(b*nchunk + chunk) * 2D].
constexpr int kLnBwdRows = 8;

template <typename T, typename Ta, int V, int NJC>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const float* __restrict__ du, const float* __restrict__ x,
                                                     const float* __restrict__ mean, const float* __restrict__ rstd,
                                                     const T* __restrict__ gamma, const float* __restrict__ mod,
                                                     int mod_off, const float* dres, int S, int D, float* dx,
                                                     Ta* __restrict__ dx_act, float* __restrict__ part) {
  constexpr int NJ = NJC > 0 ? NJC : kMaxPerLane / V;
  constexpr int RG = 2;                        // rows loaded together
  constexpr int NG = kLnBwdRows / (4 * RG);    // row groups per wave
  constexpr int CPP = 64 * kMaxPerLane / 4;    // columns per combining pass (512)
  // four waves' partials of one pass; column q * V + e of the pass at slot e * (CPP / V + 1) + q, so
  // that the writes (fixed e, consecutive q) and the reads (consecutive columns) are conflict-free
  constexpr int SLOT = CPP / V + 1;
  __shared__ float red[4][2][V * SLOT];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int b = blockIdx.y, chunk = blockIdx.x, nchunk = gridDim.x;
  const int n = NJC > 0 ? NJC : D / (64 * V);
  const float* scale = mod ? mod + (size_t)b * 6 * D + mod_off + D : nullptr;
  float pg[NJ][V], pb[NJ][V], wt[NJ][V];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    if (j < n) {
      const int c = col_of<V>(lane, j);
      if (mod) {
        ldv<V>(scale + c, wt[j]);
#pragma unroll
        for (int e = 0; e < V; ++e) wt[j][e] += 1.0f;
      } else {
        ldv<V>(gamma + c, wt[j]);
      }
    }
#pragma unroll
    for (int e = 0; e < V; ++e) { pg[j][e] = 0.f; pb[j][e] = 0.f; }
  }
#pragma unroll 1
  for (int grp = 0; grp < NG; ++grp) {
    // this wave's rows of the group (loads of both rows issued before any reduction)
    float g[RG][NJ][V], xv[RG][NJ][V], rv[RG][NJ][V];
    size_t rows[RG];
    bool ok[RG];
#pragma unroll
    for (int rr = 0; rr < RG; ++rr) {
      const int s = chunk * kLnBwdRows + wid + 4 * (grp * RG + rr);
      ok[rr] = s < S;
      rows[rr] = (size_t)b * S + (ok[rr] ? s : 0);
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if (j < n && ok[rr]) {
          ldv<V>(du + rows[rr] * D + col_of<V>(lane, j), g[rr][j]);
          ldv<V>(x + rows[rr] * D + col_of<V>(lane, j), xv[rr][j]);
          ldv<V>(dres + rows[rr] * D + col_of<V>(lane, j), rv[rr][j]);
        }
    }
#pragma unroll
    for (int rr = 0; rr < RG; ++rr) {
      if (!ok[rr]) continue;
      const size_t row = rows[rr];
      const float mu = mean[row], rs = rstd[row];
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if (j < n)
#pragma unroll
          for (int e = 0; e < V; ++e) {
            const float xh = (xv[rr][j][e] - mu) * rs;
            const float dxh = g[rr][j][e] * wt[j][e];
            s1 += dxh;
            s2 += dxh * xh;
            pg[j][e] += g[rr][j][e] * xh;
            pb[j][e] += g[rr][j][e];
            xv[rr][j][e] = xh;
          }
      const float m1 = wave_sum(s1) / (float)D, m2 = wave_sum(s2) / (float)D;
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        if (j < n) {
          const int c = col_of<V>(lane, j);
          float o[V];
#pragma unroll
          for (int e = 0; e < V; ++e) o[e] = rv[rr][j][e] + (g[rr][j][e] * wt[j][e] - m1 - xv[rr][j][e] * m2) * rs;
          stv<V>(dx + row * D + c, o);
          if (dx_act) stv<V>(dx_act + row * D + c, o);
        }
    }
  }
  // combine the four waves' partials through LDS, CPP columns per pass
  float* out = part + ((size_t)b * nchunk + chunk) * 2 * D;
  for (int c0 = 0; c0 < D; c0 += CPP) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int q = lane + 64 * j - c0 / V;   // column group (of V) within the pass
      if (j < n && q >= 0 && q < CPP / V) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          red[wid][0][e * SLOT + q] = pg[j][e];
          red[wid][1][e * SLOT + q] = pb[j][e];
        }
      }
    }
    __syncthreads();
    for (int t = threadIdx.x; t < CPP && c0 + t < D; t += 256) {
      const int sl = (t % V) * SLOT + t / V;
      out[c0 + t] = red[0][0][sl] + red[1][0][sl] + red[2][0][sl] + red[3][0][sl];
      out[D + c0 + t] = red[0][1][sl] + red[1][1][sl] + red[2][1][sl] + red[3][1][sl];
    }
  }
}

// Per-sample column sums of X (or X * Y), in chunks of kColRows rows:
// part[(b * nchunk + chunk) * N + c].  Optional per-sample column weights w[b*wstride + c].
constexpr int kColRows = 64;
template <typename TX, typename TY>
__global__ __launch_bounds__(256) void colsum_kernel(const TX* __restrict__ X, const TY* __restrict__ Y,
                                                     const float* __restrict__ w, int wstride, int S, int N,
                                                     float* __restrict__ part) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  const int chunk = blockIdx.y, b = blockIdx.z, nchunk = gridDim.y;
  if (c >= N) return;
  const int s0 = chunk * kColRows, s1 = min(S, s0 + kColRows);
  float acc = 0.f;
  // eight rows' loads in flight before their products are added, rows in ascending order
  int s = s0;
  for (; s + 8 <= s1; s += 8) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const size_t o = ((size_t)b * S + s + i) * N + c;
      v[i] = to_f32<TX>(X[o]);
      if (Y) v[i] *= to_f32<TY>(Y[o]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) acc += v[i];
  }
  for (; s < s1; ++s) {
    const size_t o = ((size_t)b * S + s) * N + c;
    float v = to_f32<TX>(X[o]);
    if (Y) v *= to_f32<TY>(Y[o]);
    acc += v;
  }
  if (w) acc *= w[(size_t)b * wstride + c];
  part[((size_t)b * nchunk + chunk) * N + c] = acc;
}

// y = T(x) elementwise (storage -> fp32, fp32 -> storage, fp32 -> activation), with an
// optional per-sample column weight (adaLN gates): y[b,s,c] = x * w[b*wstride + c].
// Eight consecutive elements per thread (n and D multiples of 8, so the eight share a row).
template <typename T>
SR_DEV void load8(const T* p, float (&v)[8]) {
  if constexpr (sizeof(T) == 4) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) { v[e] = a[e]; v[4 + e] = b[e]; }
  } else {
    const i32x4 w = *reinterpret_cast<const i32x4*>(p);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[2 * q] = __uint_as_float((uint32_t)w[q] << 16);
      v[2 * q + 1] = __uint_as_float((uint32_t)w[q] & 0xFFFF0000u);
    }
  }
}
template <typename T>
SR_DEV void store8(T* p, const float (&v)[8]) {
  if constexpr (sizeof(T) == 4) {
    *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(p + 4) = f32x4{v[4], v[5], v[6], v[7]};
  } else {
    i32x4 w;
#pragma unroll
    for (int q = 0; q < 4; ++q) w[q] = (int)f2bf2(v[2 * q], v[2 * q + 1]);
    *reinterpret_cast<i32x4*>(p) = w;
  }
}

template <typename TI, typename TO>
__global__ __launch_bounds__(256) void convert_kernel(const TI* __restrict__ x, TO* __restrict__ y, uint32_t n8,
                                                      const float* __restrict__ w, int wstride, uint32_t S,
                                                      uint32_t D, float* __restrict__ y32) {
  const uint32_t stride = gridDim.x * 256u;
  for (uint32_t i = blockIdx.x * 256u + threadIdx.x; i < n8; i += stride) {
    const size_t o = (size_t)i * 8;
    float v[8];
    load8<TI>(x + o, v);
    if (w) {
      const uint32_t row = (uint32_t)(o / D), c = (uint32_t)(o - (size_t)row * D);
      float g[8];
      load8<float>(w + (size_t)(row / S) * wstride + c, g);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] *= g[e];
    }
    store8<TO>(y + o, v);
    if (y32) store8<float>(y32 + o, v);
  }
}

// delta[b,h,s] = sum_d dO[b,s,h*hd+d] * O[b,s,h*hd+d].  One wave per token row: lane l takes
// columns 8l .. 8l+7 of each 512-column pass (16-byte loads of bf16), so a head's hd columns lie
// on hd/8 consecutive lanes, which add their partial sums with an xor butterfly (fixed order);
// the group's first lane stores.
template <typename Ta>
__global__ __launch_bounds__(256) void attn_delta_kernel(const Ta* __restrict__ dO, const Ta* __restrict__ O,
                                                         int B, int S, int H, int hd, float* __restrict__ delta) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= B * S) return;
  const int D = H * hd, G = hd / 8;   // lanes per head in a pass (4, 8 or 16)
  const int b = row / S, s = row - b * S;
  const Ta* dr = dO + (size_t)row * D;
  const Ta* orow = O + (size_t)row * D;
  for (int c0 = 0; c0 < D; c0 += 512) {
    const int c = c0 + 8 * lane;
    float acc = 0.f;
    if (c < D) {
      float a[8], o[8];
      load8<Ta>(dr + c, a);
      load8<Ta>(orow + c, o);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc += a[e] * o[e];
    }
    for (int off = G / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (c < D && (lane & (G - 1)) == 0) delta[((size_t)b * H + c / hd) * S + s] = acc;
  }
}

// Column sums of row partials, in a fixed order (deterministic):
//   v[g][c] = sum_{r < R} part[(g*R + r) * width + c]      (sum_groups: one group of G*R rows)
// columns c < half go to out_lo[g*out_stride + c], the rest to out_hi[g*out_stride + c - half].
// A block covers 64 columns with 16 row phases, combined through LDS.
__global__ __launch_bounds__(1024) void reduce_cols_kernel(const float* __restrict__ part, int R, int G, int sum_groups,
                                                           int width, int half, float* __restrict__ out_lo,
                                                           float* __restrict__ out_hi, int out_stride,
                                                           int accumulate) {
  __shared__ float red[16][65];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int c = blockIdx.x * 64 + tx;
  const int g = blockIdx.y;
  const int nrows = sum_groups ? R * G : R;
  const size_t row0 = sum_groups ? 0 : (size_t)g * R;
  float acc = 0.f;
  if (c < width) {
    // eight loads in flight per thread; the sum order (rr ascending) is fixed
    int rr = ty;
    for (; rr + 7 * 16 < nrows; rr += 8 * 16) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = part[(row0 + rr + i * 16) * width + c];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc += v[i];
    }
    for (; rr < nrows; rr += 16) acc += part[(row0 + rr) * width + c];
  }
  red[ty][tx] = acc;
  __syncthreads();
  for (int s = 8; s >= 1; s >>= 1) {
    if (ty < s) red[ty][tx] += red[ty + s][tx];
    __syncthreads();
  }
  if (ty == 0 && c < width) {   // accumulate: added to what the output holds
    float* o = c < half ? (out_lo ? out_lo + (size_t)g * out_stride + c : nullptr)
                        : (out_hi ? out_hi + (size_t)g * out_stride + c - half : nullptr);
    if (o) *o = accumulate ? *o + red[0][tx] : red[0][tx];
  }
}

// Fill with a constant (a kernel rather than a memset node, so captured graphs replay it safely).
__global__ __launch_bounds__(256) void fill_kernel(float* __restrict__ p, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) p[i] = v;
}

// ------------------------------------------------------------------------------ launchers

static inline dim3 grid1d(size_t n, int per) { return dim3((unsigned)((n + per - 1) / per)); }

hipError_t launch_ln_fwd(int dtype, const float* x, const void* gamma, const void* beta, const float* mod,
                         int mod_off, int M, int S, int D, float eps, void* y, float* mean, float* rstd,
                         hipStream_t st) {
#define SR_LNF(T, V, NJC)                                                                                    \
  SR_LAUNCH((ln_fwd_kernel<T, T, V, NJC>), grid1d(M, 4), dim3(256), 0, st, x, (const T*)gamma,      \
                     (const T*)beta, mod, mod_off, M, S, D, eps, (T*)y, mean, rstd, (const T*)nullptr, \
                     (const int32_t*)nullptr, 0, 0, (float*)nullptr)
#define SR_LNF_T(T)                                      \
  switch (D % 256 == 0 ? D / 256 : 0) {                  \
    case 1: SR_LNF(T, 4, 1); break;                      \
    case 2: SR_LNF(T, 4, 2); break;                      \
    case 4: SR_LNF(T, 4, 4); break;                      \
    case 8: SR_LNF(T, 4, 8); break;                      \
    default: if (D % 256 == 0) SR_LNF(T, 4, 0); else SR_LNF(T, 1, 0); \
  }
  if (dtype == kBF16) { SR_LNF_T(bf16_t); } else { SR_LNF_T(float); }
#undef SR_LNF_T
#undef SR_LNF
  return hipGetLastError();
}

hipError_t launch_ln_fwd_gather(int dtype, const void* xsrc, const int32_t* idx, int L, int shared, float* xcopy,
                                const void* gamma, const void* beta, const float* mod, int mod_off, int M, int S,
                                int D, float eps, void* y, float* mean, float* rstd, hipStream_t st) {
#define SR_LNG(T, V, NJC)                                                                                         \
  SR_LAUNCH((ln_fwd_kernel<T, T, V, NJC, true>), grid1d(M, 4), dim3(256), 0, st, (const float*)nullptr, \
                     (const T*)gamma, (const T*)beta, mod, mod_off, M, S, D, eps, (T*)y, mean, rstd,              \
                     (const T*)xsrc, idx, L, shared, xcopy)
#define SR_LNG_T(T)                                      \
  switch (D % 256 == 0 ? D / 256 : 0) {                  \
    case 1: SR_LNG(T, 4, 1); break;                      \
    case 2: SR_LNG(T, 4, 2); break;                      \
    case 4: SR_LNG(T, 4, 4); break;                      \
    case 8: SR_LNG(T, 4, 8); break;                      \
    default: if (D % 256 == 0) SR_LNG(T, 4, 0); else SR_LNG(T, 1, 0); \
  }
  if (dtype == kBF16) { SR_LNG_T(bf16_t); } else { SR_LNG_T(float); }
#undef SR_LNG_T
#undef SR_LNG
  return hipGetLastError();
}

hipError_t launch_ln_apply(int dtype, const float* x, const void* gamma, const void* beta, const float* mod,
                           int mod_off, int M, int S, int D, const float* mean, const float* rstd, void* y,
                           hipStream_t st) {
#define SR_LNA(T, V, NJC)                                                                                       \
  SR_LAUNCH((ln_fwd_kernel<T, T, V, NJC, false, true>), grid1d(M, 4), dim3(256), 0, st, x,            \
                     (const T*)gamma, (const T*)beta, mod, mod_off, M, S, D, 0.0f, (T*)y, const_cast<float*>(mean), \
                     const_cast<float*>(rstd), (const T*)nullptr, (const int32_t*)nullptr, 0, 0, (float*)nullptr)
#define SR_LNA_T(T)                                      \
  switch (D % 256 == 0 ? D / 256 : 0) {                  \
    case 1: SR_LNA(T, 4, 1); break;                      \
    case 2: SR_LNA(T, 4, 2); break;                      \
    case 4: SR_LNA(T, 4, 4); break;                      \
    case 8: SR_LNA(T, 4, 8); break;                      \
    default: if (D % 256 == 0) SR_LNA(T, 4, 0); else SR_LNA(T, 1, 0); \
  }
  if (dtype == kBF16) { SR_LNA_T(bf16_t); } else { SR_LNA_T(float); }
#undef SR_LNA_T
#undef SR_LNA
  return hipGetLastError();
}

int ln_bwd_chunks(int S) { return (S + kLnBwdRows - 1) / kLnBwdRows; }

hipError_t launch_ln_bwd(int dtype, const float* du, const float* x, const float* mean, const float* rstd,
                         const void* gamma, const float* mod, int mod_off, const float* dres, int B, int S, int D,
                         float* dx, void* dx_act, float* part, hipStream_t st) {
  dim3 g(ln_bwd_chunks(S), B);
#define SR_LNB(T, V, NJC)                                                                                  \
  SR_LAUNCH((ln_bwd_kernel<T, T, V, NJC>), g, dim3(256), 0, st, du, x, mean, rstd, (const T*)gamma, \
                     mod, mod_off, dres, S, D, dx, (T*)dx_act, part)
#define SR_LNB_T(T)                                      \
  switch (D % 256 == 0 ? D / 256 : 0) {                  \
    case 1: SR_LNB(T, 4, 1); break;                      \
    case 2: SR_LNB(T, 4, 2); break;                      \
    case 4: SR_LNB(T, 4, 4); break;                      \
    case 8: SR_LNB(T, 4, 8); break;                      \
    default: if (D % 256 == 0) SR_LNB(T, 4, 0); else SR_LNB(T, 1, 0); \
  }
  if (dtype == kBF16) { SR_LNB_T(bf16_t); } else { SR_LNB_T(float); }
#undef SR_LNB_T
#undef SR_LNB
  return hipGetLastError();
}

int colsum_chunks(int S) { return (S + kColRows - 1) / kColRows; }

// X type: 0 = fp32, 1 = bf16; Y likewise (Y may be null).
hipError_t launch_colsum(int xt, const void* X, int yt, const void* Y, const float* w, int wstride, int B, int S,
                         int N, float* part, hipStream_t st) {
  dim3 g((N + 255) / 256, colsum_chunks(S), B);
#define SR_COLSUM(TX, TY) \
  SR_LAUNCH((colsum_kernel<TX, TY>), g, dim3(256), 0, st, (const TX*)X, (const TY*)Y, w, wstride, S, N, part)
  if (xt == kBF16) {
    if (yt == kBF16) SR_COLSUM(bf16_t, bf16_t); else SR_COLSUM(bf16_t, float);
  } else {
    if (yt == kBF16) SR_COLSUM(float, bf16_t); else SR_COLSUM(float, float);
  }
#undef SR_COLSUM
  return hipGetLastError();
}

hipError_t launch_convert(int ti, const void* x, int to, void* y, size_t n, const float* w, int wstride, int S,
                          int D, float* y32, hipStream_t st) {
  if (n % 8 != 0 || D % 8 != 0 || n / 8 > 0xFFFFFFFFull) return hipErrorInvalidValue;
  const uint32_t n8 = (uint32_t)(n / 8);
  dim3 g((unsigned)std::min<size_t>((n8 + 255) / 256, 65536));
#define SR_CONV(TI, TO)                                                                                  \
  SR_LAUNCH((convert_kernel<TI, TO>), g, dim3(256), 0, st, (const TI*)x, (TO*)y, n8, w, wstride, \
                     (uint32_t)S, (uint32_t)D, y32)
  if (ti == kBF16) {
    if (to == kBF16) SR_CONV(bf16_t, bf16_t); else SR_CONV(bf16_t, float);
  } else {
    if (to == kBF16) SR_CONV(float, bf16_t); else SR_CONV(float, float);
  }
#undef SR_CONV
  return hipGetLastError();
}

hipError_t launch_reduce_cols(const float* part, int R, int G, int sum_groups, int width, int half, float* out_lo,
                              float* out_hi, int out_stride, hipStream_t st, int accumulate) {
  dim3 g((width + 63) / 64, sum_groups ? 1 : G);
  SR_LAUNCH(reduce_cols_kernel, g, dim3(1024), 0, st, part, R, G, sum_groups, width, half, out_lo, out_hi,
                     out_stride, accumulate);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t st) {
  dim3 g((unsigned)std::min<size_t>((n + 255) / 256, 65536));
  SR_LAUNCH(fill_kernel, g, dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_attn_delta(int dtype, const void* dO, const void* O, int B, int S, int H, int hd, float* delta,
                             hipStream_t st) {
  const size_t rows = (size_t)B * S;
  if (dtype == kBF16)
    SR_LAUNCH(attn_delta_kernel<bf16_t>, grid1d(rows, 4), dim3(256), 0, st, (const bf16_t*)dO,
                       (const bf16_t*)O, B, S, H, hd, delta);
  else
    SR_LAUNCH(attn_delta_kernel<float>, grid1d(rows, 4), dim3(256), 0, st, (const float*)dO,
                       (const float*)O, B, S, H, hd, delta);
  return hipGetLastError();
}

}  // namespace sr
