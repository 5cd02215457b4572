// Asymmetric attention of the generative block's sparse middle stage (Sec. 3.4, "Integration
// with Generative Forecasting"; App. A.1 EDM table): queries from Sq tokens (the routed ones),
// keys and values from Skv tokens (all of the conditioning sequence); per sample and head
// O = softmax(q k^T / sqrt(hd)) v over the Skv keys, and its backward.
//
// Layouts: q, O, dO, dq [B*Sq, D] (head h at columns h*hd ..); kv, dkv [B*Skv, 2D] (k of head h
// at column h*hd, v at D + h*hd); lse, delta [B, H, Sq], lse the base-2 log-sum-exp of the scaled
// scores (P = exp2(s * log2(e)/sqrt(hd) - lse)), delta = rowsum(dO * O) per head.
//
// bf16 with hd = 64 or 128 runs the MFMA attention kernels (attention.hip), which take the query
// and key/value buffers and their token counts separately.  Generic kernels (fp32 storage, or
// bf16 at hd = 32) for the rest: one thread per query (forward with online softmax, dQ) or per
// key (dK and dV, summing over the queries in order), fp32 accumulation, deterministic.
#include "common.h"
#include "sr_internal.h"

namespace sr {

template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void xattn_fwd_kernel(const Ta* __restrict__ q, const Ta* __restrict__ kv,
                                                       Ta* __restrict__ O, float* __restrict__ lse, int Sq, int Skv,
                                                       int H, int D, float sl2) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int i = blockIdx.x * 64 + threadIdx.x;
  if (i >= Sq) return;
  const size_t ldkv = 2 * (size_t)D;
  const Ta* qr = q + ((size_t)b * Sq + i) * D + hh * HDT;
  float qv[HDT], acc[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) { qv[d] = to_f32<Ta>(qr[d]); acc[d] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int j = 0; j < Skv; ++j) {
    const Ta* kr = kv + ((size_t)b * Skv + j) * ldkv + hh * HDT;
    const Ta* vr = kr + D;
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < HDT; ++d) s = fmaf(qv[d], to_f32<Ta>(kr[d]), s);
    s *= sl2;
    const float mn = fmaxf(m, s);
    const float a = exp2f(m - mn), p = exp2f(s - mn);
    l = l * a + p;
#pragma unroll
    for (int d = 0; d < HDT; ++d) acc[d] = acc[d] * a + p * to_f32<Ta>(vr[d]);
    m = mn;
  }
  Ta* orow = O + ((size_t)b * Sq + i) * D + hh * HDT;
#pragma unroll
  for (int d = 0; d < HDT; ++d) orow[d] = from_f32<Ta>(acc[d] / l);
  lse[((size_t)b * H + hh) * Sq + i] = m + log2f(l);
}

// dQ of one query: sum over the keys of dS * k, dS = P (dP - delta), dP = dO . v.
template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void xattn_bwd_dq_kernel(const Ta* __restrict__ q, const Ta* __restrict__ kv,
                                                          const Ta* __restrict__ dO, const float* __restrict__ lse,
                                                          const float* __restrict__ delta, Ta* __restrict__ dq, int Sq,
                                                          int Skv, int H, int D, float sl2, float scale) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int i = blockIdx.x * 64 + threadIdx.x;
  if (i >= Sq) return;
  const size_t ldkv = 2 * (size_t)D;
  const size_t row = (size_t)b * Sq + i;
  float qv[HDT], dov[HDT], acc[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) {
    qv[d] = to_f32<Ta>(q[row * D + hh * HDT + d]);
    dov[d] = to_f32<Ta>(dO[row * D + hh * HDT + d]);
    acc[d] = 0.f;
  }
  const float L2 = lse[((size_t)b * H + hh) * Sq + i], dl = delta[((size_t)b * H + hh) * Sq + i];
  for (int j = 0; j < Skv; ++j) {
    const Ta* kr = kv + ((size_t)b * Skv + j) * ldkv + hh * HDT;
    const Ta* vr = kr + D;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int d = 0; d < HDT; ++d) {
      s = fmaf(qv[d], to_f32<Ta>(kr[d]), s);
      dp = fmaf(dov[d], to_f32<Ta>(vr[d]), dp);
    }
    const float ds = exp2f(s * sl2 - L2) * (dp - dl);
#pragma unroll
    for (int d = 0; d < HDT; ++d) acc[d] = fmaf(ds, to_f32<Ta>(kr[d]), acc[d]);
  }
#pragma unroll
  for (int d = 0; d < HDT; ++d) dq[row * D + hh * HDT + d] = from_f32<Ta>(acc[d] * scale);
}

// dK and dV of one key: sums over the queries of dS * q and P * dO.
template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void xattn_bwd_dkv_kernel(const Ta* __restrict__ q, const Ta* __restrict__ kv,
                                                           const Ta* __restrict__ dO, const float* __restrict__ lse,
                                                           const float* __restrict__ delta, Ta* __restrict__ dkv,
                                                           int Sq, int Skv, int H, int D, float sl2, float scale) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int j = blockIdx.x * 64 + threadIdx.x;
  if (j >= Skv) return;
  const size_t ldkv = 2 * (size_t)D;
  const size_t krow = ((size_t)b * Skv + j) * ldkv + hh * HDT;
  float kvv[HDT], vv[HDT], dk[HDT], dv[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) {
    kvv[d] = to_f32<Ta>(kv[krow + d]);
    vv[d] = to_f32<Ta>(kv[krow + D + d]);
    dk[d] = 0.f;
    dv[d] = 0.f;
  }
  for (int i = 0; i < Sq; ++i) {
    const Ta* qr = q + ((size_t)b * Sq + i) * D + hh * HDT;
    const Ta* dr = dO + ((size_t)b * Sq + i) * D + hh * HDT;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int d = 0; d < HDT; ++d) {
      s = fmaf(to_f32<Ta>(qr[d]), kvv[d], s);
      dp = fmaf(to_f32<Ta>(dr[d]), vv[d], dp);
    }
    const size_t st = ((size_t)b * H + hh) * Sq + i;
    const float p = exp2f(s * sl2 - lse[st]);
    const float ds = p * (dp - delta[st]);
#pragma unroll
    for (int d = 0; d < HDT; ++d) {
      dv[d] = fmaf(p, to_f32<Ta>(dr[d]), dv[d]);
      dk[d] = fmaf(ds, to_f32<Ta>(qr[d]), dk[d]);
    }
  }
#pragma unroll
  for (int d = 0; d < HDT; ++d) {
    dkv[krow + d] = from_f32<Ta>(dk[d] * scale);
    dkv[krow + D + d] = from_f32<Ta>(dv[d]);
  }
}

static inline float xattn_sl2(int hd) { return 1.4426950408889634f / sqrtf((float)hd); }

template <typename Ta>
static hipError_t xfwd(const Ta* q, const Ta* kv, Ta* O, float* lse, int B, int Sq, int Skv, int H, int D,
                       hipStream_t st) {
  const int hd = D / H;
  dim3 g((Sq + 63) / 64, H, B);
  const float sl2 = xattn_sl2(hd);
  if (hd == 32) SR_LAUNCH((xattn_fwd_kernel<Ta, 32>), g, dim3(64), 0, st, q, kv, O, lse, Sq, Skv, H, D, sl2);
  else if (hd == 64) SR_LAUNCH((xattn_fwd_kernel<Ta, 64>), g, dim3(64), 0, st, q, kv, O, lse, Sq, Skv, H, D, sl2);
  else SR_LAUNCH((xattn_fwd_kernel<Ta, 128>), g, dim3(64), 0, st, q, kv, O, lse, Sq, Skv, H, D, sl2);
  return hipGetLastError();
}

template <typename Ta>
static hipError_t xbwd(const Ta* q, const Ta* kv, const Ta* dO, const float* lse, const float* delta, Ta* dq,
                       Ta* dkv, int B, int Sq, int Skv, int H, int D, hipStream_t st) {
  const int hd = D / H;
  dim3 gq((Sq + 63) / 64, H, B), gk((Skv + 63) / 64, H, B);
  const float sl2 = xattn_sl2(hd), sc = 1.0f / sqrtf((float)hd);
#define SR_XB(HDV)                                                                                                 \
  SR_LAUNCH((xattn_bwd_dq_kernel<Ta, HDV>), gq, dim3(64), 0, st, q, kv, dO, lse, delta, dq, Sq, Skv, H, D, \
                     sl2, sc);                                                                                     \
  SR_LAUNCH((xattn_bwd_dkv_kernel<Ta, HDV>), gk, dim3(64), 0, st, q, kv, dO, lse, delta, dkv, Sq, Skv, H, \
                     D, sl2, sc)
  if (hd == 32) { SR_XB(32); } else if (hd == 64) { SR_XB(64); } else { SR_XB(128); }
#undef SR_XB
  return hipGetLastError();
}

hipError_t launch_xattn_fwd(int dtype, const void* q, const void* kv, void* O, float* lse, int B, int Sq, int Skv,
                            int H, int D, hipStream_t st) {
  if (attn_uses_mfma(dtype, D / H))
    return launch_attn_fwd_mfma((const bf16_t*)q, D, (const bf16_t*)kv, 2 * D, (uint32_t)((size_t)B * Skv * 2 * D),
                                (bf16_t*)O, lse, B, Sq, Skv, H, D, st);
  if (dtype == kBF16) return xfwd((const bf16_t*)q, (const bf16_t*)kv, (bf16_t*)O, lse, B, Sq, Skv, H, D, st);
  return xfwd((const float*)q, (const float*)kv, (float*)O, lse, B, Sq, Skv, H, D, st);
}

hipError_t launch_xattn_bwd(int dtype, const void* q, const void* kv, const void* O, const void* dO, const float* lse,
                            float* delta, void* dq, void* dkv, int B, int Sq, int Skv, int H, int D, hipStream_t st) {
  hipError_t e = launch_attn_delta(dtype, dO, O, B, Sq, H, D / H, delta, st);
  if (e != hipSuccess) return e;
  if (attn_uses_mfma(dtype, D / H)) {
    const bf16_t *qb = (const bf16_t*)q, *kvb = (const bf16_t*)kv, *dOb = (const bf16_t*)dO;
    e = launch_attn_dkv_mfma(qb, D, (uint32_t)((size_t)B * Sq * D), kvb, 2 * D, dOb, lse, delta, (bf16_t*)dkv, 2 * D, B,
                             Sq, Skv, H, D, st);
    if (e != hipSuccess) return e;
    return launch_attn_dq_mfma(qb, D, kvb, 2 * D, (uint32_t)((size_t)B * Skv * 2 * D), dOb, lse, delta, (bf16_t*)dq, D,
                               B, Sq, Skv, H, D, st);
  }
  if (dtype == kBF16)
    return xbwd((const bf16_t*)q, (const bf16_t*)kv, (const bf16_t*)dO, lse, delta, (bf16_t*)dq, (bf16_t*)dkv, B, Sq,
                Skv, H, D, st);
  return xbwd((const float*)q, (const float*)kv, (const float*)dO, lse, delta, (float*)dq, (float*)dkv, B, Sq, Skv, H,
              D, st);
}

}  // namespace sr
