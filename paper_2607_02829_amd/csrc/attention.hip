// Multi-head self-attention of the block (Sec. 3.3): per sample and head,
// O = softmax(q k^T / sqrt(hd)) v over all S tokens (no mask), and its backward.
//
// Layouts: qkv is token-major [B*S, 3D] (q at column h*hd, k at D + h*hd, v at
// 2D + h*hd); O and dO are [B*S, D]; dqkv mirrors qkv.  lse[b,h,s] is the base-2
// log-sum-exp of the scaled scores, so P = exp2(s * log2(e)/sqrt(hd) - lse).
//
// MFMA kernels (hd = 64, bf16, v_mfma_f32_32x32x16_bf16):
//  * forward: a wave owns 32 queries and computes S^T = K Q^T for 64-key LDS
//    tiles, so each lane holds one query's scores and the online-softmax state
//    (running max, partial sum) is per lane; one xor-32 exchange per tile gives
//    the row max.  O^T += V^T P^T reuses the score registers directly as the B
//    operand (the k order inside an MFMA is free as long as A and B agree), with
//    V staged transposed in LDS.  The S x S score matrix is never stored.
//  * backward dK/dV: a wave owns 32 keys; for 64-query tiles it forms
//    S = Q K^T and dP = dO V^T (key per lane), P = exp2(S c - lse),
//    dS = P (dP - delta), then dV^T += dO^T P and dK^T += Q^T dS.
//  * backward dQ: a wave owns 32 queries; S^T, dP^T per 64-key tile and
//    dQ^T += K^T dS^T.
// Two backward passes (instead of atomics) keep the result deterministic.
//
// Generic kernels (any storage type, hd in {32, 64, 128}): one thread per row,
// online softmax over keys, fp32 throughout.
#include <type_traits>

#include "common.h"
#include "profile.h"
#include "sr_internal.h"

namespace sr {

constexpr int HD = 64;
constexpr int AP = HD + 8;   // padded LDS row (bf16)
constexpr int QW = 128;      // rows (queries or keys) per workgroup, 32 per wave
constexpr int KT = 64;       // tile of the streamed dimension

SR_DEV bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
  return z;
}

SR_DEV bf16x8 ld8(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

// A fragment whose k order matches a score fragment: elements 0..3 from p[4*h],
// elements 4..7 from p[8 + 4*h].
SR_DEV bf16x8 ld_perm(const bf16_t* p, int h) {
  i32x2 lo = *reinterpret_cast<const i32x2*>(p + 4 * h);
  i32x2 hi = *reinterpret_cast<const i32x2*>(p + 8 + 4 * h);
  i32x4 v;
  v[0] = lo[0]; v[1] = lo[1]; v[2] = hi[0]; v[3] = hi[1];
  return *reinterpret_cast<bf16x8*>(&v);
}

SR_DEV f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) { return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0); }

// 2^x on the hardware unit directly: the softmax arguments are <= 0 (or -inf), where the
// unscaled instruction is accurate to ~1 ulp and flushes tiny results to zero.
SR_DEV float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

SR_DEV void zero16(f32x16& a) {
#pragma unroll
  for (int r = 0; r < 16; ++r) a[r] = 0.f;
}

// A 64 x 64 tile of one head (rows r0.., head columns), moved by 256 threads: thread
// (dg = tid % 16, rg = tid / 16) holds rows 4rg..4rg+3, columns 4dg..4dg+3 in registers, so
// one global read can be written to LDS row-major, transposed, or both.
struct Tile4 {
  i32x2 v[4];
};

// Rows past the sample's S tokens are read without a guard: they belong to the next
// sample (finite values that the callers neutralise: keys get a -inf score, queries an
// infinite LSE) or lie past the tensor, where the buffer load returns zero.
// `base` is the byte offset of (row 0, column 0 of the head) inside the tensor of `rs`.
SR_DEV void t4_load(Tile4& t, __amdgpu_buffer_rsrc_t rs, uint32_t base, uint32_t ld, int r0) {
  const int dg = threadIdx.x & 15, rg = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    t.v[i] = buf_load8(rs, base + ((uint32_t)(r0 + rg * 4 + i) * ld + (uint32_t)dg * 4u) * 2u);
}

// lds[row][d]
SR_DEV void t4_rows(const Tile4& t, bf16_t* lds) {
  const int dg = threadIdx.x & 15, rg = threadIdx.x >> 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<i32x2*>(lds + (rg * 4 + i) * AP + dg * 4) = t.v[i];
}

// lds[d][row]
SR_DEV void t4_cols(const Tile4& t, bf16_t* lds) {
  const int dg = threadIdx.x & 15, rg = threadIdx.x >> 4;
  const uint16_t* e0 = reinterpret_cast<const uint16_t*>(&t.v[0]);
  const uint16_t* e1 = reinterpret_cast<const uint16_t*>(&t.v[1]);
  const uint16_t* e2 = reinterpret_cast<const uint16_t*>(&t.v[2]);
  const uint16_t* e3 = reinterpret_cast<const uint16_t*>(&t.v[3]);
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    i32x2 w;
    w[0] = (int)((uint32_t)e0[c] | ((uint32_t)e1[c] << 16));
    w[1] = (int)((uint32_t)e2[c] | ((uint32_t)e3[c] << 16));
    *reinterpret_cast<i32x2*>(lds + (dg * 4 + c) * AP + rg * 4) = w;
  }
}

// Write a wave's 32 x 64 result (held transposed: acc[db][r] = X[d][row]) to LDS
// stage[row_local][d], scaled.
SR_DEV void stage_t(bf16_t* stage, const f32x16 acc[2], float mul, int wid, int lane) {
  const int l32 = lane & 31, h32 = lane >> 5;
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int d = db * 32 + 8 * (r >> 2) + 4 * h32 + (r & 3);
      stage[(wid * 32 + l32) * AP + d] = f2bf(acc[db][r] * mul);
    }
}

// Copy the 128 x 64 staged tile to rows r0.. of dst (column block of one head).
SR_DEV void unstage(const bf16_t* stage, bf16_t* dst, size_t ld, int r0, int S) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = threadIdx.x + 256 * i;
    const int row = c >> 3, kc = c & 7;
    if (r0 + row < S)
      *reinterpret_cast<i32x4*>(dst + (size_t)(r0 + row) * ld + kc * 8) =
          *reinterpret_cast<const i32x4*>(stage + row * AP + kc * 8);
  }
}

// All three MFMA kernels stream 64-row tiles through two LDS stages: while tile t is
// consumed from one stage, tile t+1 is already in flight from global memory into
// registers and is written into the other stage afterwards (one barrier per tile).

// ------------------------------------------------------------------------------ forward

__global__ __launch_bounds__(256, 2) void attn_fwd_mfma(const bf16_t* __restrict__ qkv, bf16_t* __restrict__ O,
                                                     float* __restrict__ lse, int S, int H, int D, float sl2) {
  constexpr int ST = 2 * KT * AP;   // one stage: Ks [key][d], Vt [d][key]
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * ST];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const int b = blockIdx.z, hh = blockIdx.y;
  const size_t ld = 3 * (size_t)D;
  const bf16_t* base = qkv + (size_t)b * S * ld;
  const bf16_t* qp = base + hh * HD;
  const int myq = blockIdx.x * QW + wid * 32 + l32;
  const int ntiles = (S + KT - 1) / KT;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qkv, (uint32_t)((size_t)gridDim.z * S * ld * 2));
  const uint32_t kbase = (uint32_t)(((size_t)b * S * ld + D + hh * HD) * 2);
  const uint32_t vbase = kbase + (uint32_t)D * 2u;

  bf16x8 qf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) qf[ks] = myq < S ? ld8(qp + (size_t)myq * ld + ks * 16 + 8 * h32) : zero8();

  Tile4 kr, vr;
  t4_load(kr, rq, kbase, (uint32_t)ld, 0);
  t4_load(vr, rq, vbase, (uint32_t)ld, 0);
  t4_rows(kr, smem);
  t4_cols(vr, smem + KT * AP);
  __syncthreads();

  f32x16 o[2];
  zero16(o[0]); zero16(o[1]);
  float m_run = -INFINITY, l_run = 0.f;   // running max of the raw scores, partial sum

  // one key tile: prefetch the next, consume this one from LDS, stage the next
  auto step = [&](int t, auto ragged) {
    const int k0 = t * KT;
    const bool more = t + 1 < ntiles;
    if (more) {
      t4_load(kr, rq, kbase, (uint32_t)ld, k0 + KT);
      t4_load(vr, rq, vbase, (uint32_t)ld, k0 + KT);
    }
    const bf16_t* Ks = smem + (t & 1) * ST;
    const bf16_t* Vt = Ks + KT * AP;
    {
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        zero16(s[kb]);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) s[kb] = mfma(ld8(Ks + (kb * 32 + l32) * AP + ks * 16 + 8 * h32), qf[ks], s[kb]);
      }
      if constexpr (decltype(ragged)::value) {   // last tile: keys past S do not exist
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (k0 + kb * 32 + 8 * (r >> 2) + 4 * h32 + (r & 3) >= S) s[kb][r] = -INFINITY;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = ex2((m_run - m_new) * sl2);
      const float nm = -m_new * sl2;
      float psum = 0.f;
      bf16x8 pb[2][2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = ex2(fmaf(s[kb][r], sl2, nm));
          psum += p;
          pb[kb][r >> 3][r & 7] = (__bf16)p;
        }
      l_run = l_run * alpha + psum;
      m_run = m_new;
      if (__ballot(alpha != 1.0f)) {
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      }
#pragma unroll
      for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int kk = 0; kk < 2; ++kk)
            o[db] = mfma(ld_perm(Vt + (db * 32 + l32) * AP + kb * 32 + kk * 16, h32), pb[kb][kk], o[db]);
    }
    if (more) {
      bf16_t* nx = smem + ((t + 1) & 1) * ST;
      t4_rows(kr, nx);
      t4_cols(vr, nx + KT * AP);
    }
    __syncthreads();
  };
  // full tiles, then the ragged last tile (masking only there)
  for (int t = 0; t < S / KT; ++t) step(t, std::false_type{});
  if (S % KT) step(S / KT, std::true_type{});
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (h32 == 0 && myq < S) lse[((size_t)b * H + hh) * S + myq] = m_run * sl2 + log2f(l_tot);
  stage_t(smem, o, 1.0f / l_tot, wid, lane);
  __syncthreads();
  unstage(smem, O + (size_t)b * S * D + hh * HD, D, blockIdx.x * QW, S);
}

// ------------------------------------------------------------------------------ backward dK, dV

__global__ __launch_bounds__(256, 2) void attn_bwd_dkv_mfma(const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ dO,
                                                         const float* __restrict__ lse, const float* __restrict__ delta,
                                                         bf16_t* __restrict__ dqkv, int S, int H, int D, float sl2,
                                                         float scale) {
  constexpr int STB = 4 * KT * AP;                 // bf16 per stage: Qs, dOs [q][d]; Qt, dOt [d][q]
  constexpr int STF = 2 * KT;                      // floats per stage: lse, delta of the tile's rows
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * STB];
  __shared__ float fsm[2 * STF];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const int b = blockIdx.z, hh = blockIdx.y;
  const size_t ld = 3 * (size_t)D;
  const bf16_t* base = qkv + (size_t)b * S * ld;
  const bf16_t* qp = base + hh * HD;
  const bf16_t* kp = base + D + hh * HD;
  const bf16_t* vp = base + 2 * D + hh * HD;
  const bf16_t* dop = dO + (size_t)b * S * D + hh * HD;
  const float* lse_b = lse + ((size_t)b * H + hh) * S;
  const float* dl_b = delta + ((size_t)b * H + hh) * S;
  const int mykey = blockIdx.x * QW + wid * 32 + l32;
  const int ntiles = (S + KT - 1) / KT;

  bf16x8 kf[4], vf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    kf[ks] = mykey < S ? ld8(kp + (size_t)mykey * ld + ks * 16 + 8 * h32) : zero8();
    vf[ks] = mykey < S ? ld8(vp + (size_t)mykey * ld + ks * 16 + 8 * h32) : zero8();
  }
  f32x16 dv[2], dk[2];
  zero16(dv[0]); zero16(dv[1]); zero16(dk[0]); zero16(dk[1]);

  Tile4 qr, dr;
  float lr = INFINITY, drl = 0.f;   // this thread's row statistic (threads < 64)
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qkv, (uint32_t)((size_t)gridDim.z * S * ld * 2));
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(dO, (uint32_t)((size_t)gridDim.z * S * D * 2));
  const uint32_t qbase = (uint32_t)(((size_t)b * S * ld + hh * HD) * 2);
  const uint32_t dbase = (uint32_t)(((size_t)b * S * D + hh * HD) * 2);
  auto fetch = [&](int q0) {
    t4_load(qr, rq, qbase, (uint32_t)ld, q0);
    t4_load(dr, rd, dbase, (uint32_t)D, q0);
    if (threadIdx.x < KT) {
      const int q = q0 + threadIdx.x;
      lr = q < S ? lse_b[q] : INFINITY;   // rows past S: P = 0
      drl = q < S ? dl_b[q] : 0.f;
    }
  };
  auto put = [&](int s) {
    bf16_t* st = smem + s * STB;
    t4_rows(qr, st);
    t4_rows(dr, st + KT * AP);
    t4_cols(qr, st + 2 * KT * AP);
    t4_cols(dr, st + 3 * KT * AP);
    if (threadIdx.x < KT) {
      fsm[s * STF + threadIdx.x] = lr;
      fsm[s * STF + KT + threadIdx.x] = drl;
    }
  };
  fetch(0);
  put(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const bool more = t + 1 < ntiles;
    if (more) fetch((t + 1) * KT);
    const bf16_t* Qs = smem + (t & 1) * STB;
    const bf16_t* dOs = Qs + KT * AP;
    const bf16_t* Qt = Qs + 2 * KT * AP;
    const bf16_t* dOt = Qs + 3 * KT * AP;
    const float* lse_s = fsm + (t & 1) * STF;
    const float* dl_s = lse_s + KT;
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      f32x16 s, dp;
      zero16(s); zero16(dp);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        s = mfma(ld8(Qs + (qb * 32 + l32) * AP + ks * 16 + 8 * h32), kf[ks], s);
        dp = mfma(ld8(dOs + (qb * 32 + l32) * AP + ks * 16 + 8 * h32), vf[ks], dp);
      }
      bf16x8 pb[2], sb[2];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ql = qb * 32 + 8 * (r >> 2) + 4 * h32 + (r & 3);
        const float p = ex2(fmaf(s[r], sl2, -lse_s[ql]));
        const float ds = p * (dp[r] - dl_s[ql]);
        pb[r >> 3][r & 7] = (__bf16)p;
        sb[r >> 3][r & 7] = (__bf16)ds;
      }
#pragma unroll
      for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          dv[db] = mfma(ld_perm(dOt + (db * 32 + l32) * AP + qb * 32 + kk * 16, h32), pb[kk], dv[db]);
          dk[db] = mfma(ld_perm(Qt + (db * 32 + l32) * AP + qb * 32 + kk * 16, h32), sb[kk], dk[db]);
        }
    }
    if (more) put((t + 1) & 1);
    __syncthreads();
  }
  bf16_t* out = dqkv + (size_t)b * S * ld;
  stage_t(smem, dk, scale, wid, lane);
  __syncthreads();
  unstage(smem, out + D + hh * HD, ld, blockIdx.x * QW, S);
  __syncthreads();
  stage_t(smem, dv, 1.0f, wid, lane);
  __syncthreads();
  unstage(smem, out + 2 * D + hh * HD, ld, blockIdx.x * QW, S);
}

// ------------------------------------------------------------------------------ backward dQ

__global__ __launch_bounds__(256, 2) void attn_bwd_dq_mfma(const bf16_t* __restrict__ qkv, const bf16_t* __restrict__ dO,
                                                        const float* __restrict__ lse, const float* __restrict__ delta,
                                                        bf16_t* __restrict__ dqkv, int S, int H, int D, float sl2,
                                                        float scale) {
  constexpr int ST = 3 * KT * AP;   // one stage: Ks, Vs [key][d]; Kt [d][key]
  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * ST];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const int b = blockIdx.z, hh = blockIdx.y;
  const size_t ld = 3 * (size_t)D;
  const bf16_t* base = qkv + (size_t)b * S * ld;
  const bf16_t* qp = base + hh * HD;
  const bf16_t* kp = base + D + hh * HD;
  const bf16_t* vp = base + 2 * D + hh * HD;
  const bf16_t* dop = dO + (size_t)b * S * D + hh * HD;
  const int myq = blockIdx.x * QW + wid * 32 + l32;
  const int ntiles = (S + KT - 1) / KT;

  bf16x8 qf[4], df[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    qf[ks] = myq < S ? ld8(qp + (size_t)myq * ld + ks * 16 + 8 * h32) : zero8();
    df[ks] = myq < S ? ld8(dop + (size_t)myq * D + ks * 16 + 8 * h32) : zero8();
  }
  const float nlse = myq < S ? -lse[((size_t)b * H + hh) * S + myq] : -INFINITY;
  const float dl_q = myq < S ? delta[((size_t)b * H + hh) * S + myq] : 0.f;
  f32x16 dq[2];
  zero16(dq[0]); zero16(dq[1]);

  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qkv, (uint32_t)((size_t)gridDim.z * S * ld * 2));
  const uint32_t kbase = (uint32_t)(((size_t)b * S * ld + D + hh * HD) * 2);
  const uint32_t vbase = kbase + (uint32_t)D * 2u;
  Tile4 kr, vr;
  t4_load(kr, rq, kbase, (uint32_t)ld, 0);
  t4_load(vr, rq, vbase, (uint32_t)ld, 0);
  t4_rows(kr, smem);
  t4_rows(vr, smem + KT * AP);
  t4_cols(kr, smem + 2 * KT * AP);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int k0 = t * KT;
    const bool more = t + 1 < ntiles;
    if (more) {
      t4_load(kr, rq, kbase, (uint32_t)ld, k0 + KT);
      t4_load(vr, rq, vbase, (uint32_t)ld, k0 + KT);
    }
    const bf16_t* Ks = smem + (t & 1) * ST;
    const bf16_t* Vs = Ks + KT * AP;
    const bf16_t* Kt = Ks + 2 * KT * AP;
    const bool ragged = k0 + KT > S;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16 s, dp;
      zero16(s); zero16(dp);
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        s = mfma(ld8(Ks + (kb * 32 + l32) * AP + ks * 16 + 8 * h32), qf[ks], s);
        dp = mfma(ld8(Vs + (kb * 32 + l32) * AP + ks * 16 + 8 * h32), df[ks], dp);
      }
      if (ragged) {   // last tile: keys past S do not exist
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (k0 + kb * 32 + 8 * (r >> 2) + 4 * h32 + (r & 3) >= S) s[r] = -INFINITY;
      }
      bf16x8 sb[2];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = ex2(fmaf(s[r], sl2, nlse));
        sb[r >> 3][r & 7] = (__bf16)(p * (dp[r] - dl_q));
      }
#pragma unroll
      for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk)
          dq[db] = mfma(ld_perm(Kt + (db * 32 + l32) * AP + kb * 32 + kk * 16, h32), sb[kk], dq[db]);
    }
    if (more) {
      bf16_t* nx = smem + ((t + 1) & 1) * ST;
      t4_rows(kr, nx);
      t4_rows(vr, nx + KT * AP);
      t4_cols(kr, nx + 2 * KT * AP);
    }
    __syncthreads();
  }
  stage_t(smem, dq, scale, wid, lane);
  __syncthreads();
  unstage(smem, dqkv + (size_t)b * S * ld + hh * HD, ld, blockIdx.x * QW, S);
}

// ------------------------------------------------------------------------------ generic kernels

template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void attn_fwd_simple(const Ta* __restrict__ qkv, Ta* __restrict__ O,
                                                      float* __restrict__ lse, int S, int H, int D, float sl2) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int q = blockIdx.x * 64 + threadIdx.x;
  if (q >= S) return;
  const size_t ld = 3 * (size_t)D;
  const Ta* base = qkv + (size_t)b * S * ld;
  float qv[HDT], acc[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) { qv[d] = to_f32<Ta>(base[(size_t)q * ld + hh * HDT + d]); acc[d] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int k = 0; k < S; ++k) {
    const Ta* kr = base + (size_t)k * ld + D + hh * HDT;
    const Ta* vr = base + (size_t)k * ld + 2 * D + hh * HDT;
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
  Ta* orow = O + ((size_t)b * S + q) * D + hh * HDT;
#pragma unroll
  for (int d = 0; d < HDT; ++d) orow[d] = from_f32<Ta>(acc[d] / l);
  lse[((size_t)b * H + hh) * S + q] = m + log2f(l);
}

template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void attn_bwd_dq_simple(const Ta* __restrict__ qkv, const Ta* __restrict__ dO,
                                                         const float* __restrict__ lse, const float* __restrict__ delta,
                                                         Ta* __restrict__ dqkv, int S, int H, int D, float sl2,
                                                         float scale) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int q = blockIdx.x * 64 + threadIdx.x;
  if (q >= S) return;
  const size_t ld = 3 * (size_t)D;
  const Ta* base = qkv + (size_t)b * S * ld;
  float qv[HDT], dov[HDT], acc[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) {
    qv[d] = to_f32<Ta>(base[(size_t)q * ld + hh * HDT + d]);
    dov[d] = to_f32<Ta>(dO[((size_t)b * S + q) * D + hh * HDT + d]);
    acc[d] = 0.f;
  }
  const float L2 = lse[((size_t)b * H + hh) * S + q], dl = delta[((size_t)b * H + hh) * S + q];
  for (int k = 0; k < S; ++k) {
    const Ta* kr = base + (size_t)k * ld + D + hh * HDT;
    const Ta* vr = base + (size_t)k * ld + 2 * D + hh * HDT;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int d = 0; d < HDT; ++d) {
      s = fmaf(qv[d], to_f32<Ta>(kr[d]), s);
      dp = fmaf(dov[d], to_f32<Ta>(vr[d]), dp);
    }
    const float p = exp2f(s * sl2 - L2);
    const float ds = p * (dp - dl);
#pragma unroll
    for (int d = 0; d < HDT; ++d) acc[d] = fmaf(ds, to_f32<Ta>(kr[d]), acc[d]);
  }
  Ta* out = dqkv + ((size_t)b * S + q) * ld + hh * HDT;
#pragma unroll
  for (int d = 0; d < HDT; ++d) out[d] = from_f32<Ta>(acc[d] * scale);
}

template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void attn_bwd_dkv_simple(const Ta* __restrict__ qkv, const Ta* __restrict__ dO,
                                                          const float* __restrict__ lse, const float* __restrict__ delta,
                                                          Ta* __restrict__ dqkv, int S, int H, int D, float sl2,
                                                          float scale) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int k = blockIdx.x * 64 + threadIdx.x;
  if (k >= S) return;
  const size_t ld = 3 * (size_t)D;
  const Ta* base = qkv + (size_t)b * S * ld;
  float kv[HDT], vv[HDT], dk[HDT], dv[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) {
    kv[d] = to_f32<Ta>(base[(size_t)k * ld + D + hh * HDT + d]);
    vv[d] = to_f32<Ta>(base[(size_t)k * ld + 2 * D + hh * HDT + d]);
    dk[d] = 0.f; dv[d] = 0.f;
  }
  for (int q = 0; q < S; ++q) {
    const Ta* qr = base + (size_t)q * ld + hh * HDT;
    const Ta* dr = dO + ((size_t)b * S + q) * D + hh * HDT;
    float s = 0.f, dp = 0.f;
#pragma unroll
    for (int d = 0; d < HDT; ++d) {
      s = fmaf(to_f32<Ta>(qr[d]), kv[d], s);
      dp = fmaf(to_f32<Ta>(dr[d]), vv[d], dp);
    }
    const float p = exp2f(s * sl2 - lse[((size_t)b * H + hh) * S + q]);
    const float ds = p * (dp - delta[((size_t)b * H + hh) * S + q]);
#pragma unroll
    for (int d = 0; d < HDT; ++d) {
      dv[d] = fmaf(p, to_f32<Ta>(dr[d]), dv[d]);
      dk[d] = fmaf(ds, to_f32<Ta>(qr[d]), dk[d]);
    }
  }
  Ta* out = dqkv + ((size_t)b * S + k) * ld + hh * HDT;
#pragma unroll
  for (int d = 0; d < HDT; ++d) {
    out[D + d] = from_f32<Ta>(dk[d] * scale);
    out[2 * D + d] = from_f32<Ta>(dv[d]);
  }
}

// ------------------------------------------------------------------------------ launchers

static inline float attn_sl2(int hd) { return 1.4426950408889634f / sqrtf((float)hd); }

bool attn_uses_mfma(int dtype, int hd) { return dtype == kBF16 && hd == HD; }

template <typename Ta>
static hipError_t fwd_simple(const Ta* qkv, Ta* O, float* lse, int B, int S, int H, int D, int hd, hipStream_t st) {
  dim3 g((S + 63) / 64, H, B);
  const float sl2 = attn_sl2(hd);
  if (hd == 32) hipLaunchKernelGGL((attn_fwd_simple<Ta, 32>), g, dim3(64), 0, st, qkv, O, lse, S, H, D, sl2);
  else if (hd == 64) hipLaunchKernelGGL((attn_fwd_simple<Ta, 64>), g, dim3(64), 0, st, qkv, O, lse, S, H, D, sl2);
  else hipLaunchKernelGGL((attn_fwd_simple<Ta, 128>), g, dim3(64), 0, st, qkv, O, lse, S, H, D, sl2);
  return hipGetLastError();
}

template <typename Ta>
static hipError_t bwd_simple(const Ta* qkv, const Ta* dO, const float* lse, const float* delta, Ta* dqkv, int B,
                             int S, int H, int D, int hd, hipStream_t st) {
  dim3 g((S + 63) / 64, H, B);
  const float sl2 = attn_sl2(hd), sc = 1.0f / sqrtf((float)hd);
#define SR_ABS(HDV)                                                                                              \
  hipLaunchKernelGGL((attn_bwd_dq_simple<Ta, HDV>), g, dim3(64), 0, st, qkv, dO, lse, delta, dqkv, S, H, D, sl2, sc); \
  hipLaunchKernelGGL((attn_bwd_dkv_simple<Ta, HDV>), g, dim3(64), 0, st, qkv, dO, lse, delta, dqkv, S, H, D, sl2, sc)
  if (hd == 32) { SR_ABS(32); } else if (hd == 64) { SR_ABS(64); } else { SR_ABS(128); }
#undef SR_ABS
  return hipGetLastError();
}

hipError_t launch_attn_fwd(int dtype, const void* qkv, void* O, float* lse, int B, int S, int H, int D,
                           hipStream_t st) {
  const int hd = D / H;
  if (attn_uses_mfma(dtype, hd)) {
    dim3 g((S + QW - 1) / QW, H, B);
    hipLaunchKernelGGL(attn_fwd_mfma, g, dim3(256), 0, st, (const bf16_t*)qkv, (bf16_t*)O, lse, S, H, D,
                       attn_sl2(hd));
    return hipGetLastError();
  }
  if (dtype == kBF16) return fwd_simple((const bf16_t*)qkv, (bf16_t*)O, lse, B, S, H, D, hd, st);
  return fwd_simple((const float*)qkv, (float*)O, lse, B, S, H, D, hd, st);
}

hipError_t launch_attn_bwd(int dtype, const void* qkv, const void* dO, const float* lse, const float* delta,
                           void* dqkv, int B, int S, int H, int D, hipStream_t st) {
  const int hd = D / H;
  if (attn_uses_mfma(dtype, hd)) {
    dim3 g((S + QW - 1) / QW, H, B);
    const float sl2 = attn_sl2(hd), sc = 1.0f / sqrtf((float)hd);
    const double units = 2.0 * B * (double)S * S * D;   // one S x S x hd product over all heads
    {
      // algorithmic: dP, dV, dK (the recomputed scores are not counted)
      ProfScope ps("attn_bwd_dkv", 3 * units, (double)B * S * D * 2 * 6, st);
      hipLaunchKernelGGL(attn_bwd_dkv_mfma, g, dim3(256), 0, st, (const bf16_t*)qkv, (const bf16_t*)dO, lse, delta,
                         (bf16_t*)dqkv, S, H, D, sl2, sc);
    }
    {
      ProfScope ps("attn_bwd_dq", units, (double)B * S * D * 2 * 5, st);
      hipLaunchKernelGGL(attn_bwd_dq_mfma, g, dim3(256), 0, st, (const bf16_t*)qkv, (const bf16_t*)dO, lse, delta,
                         (bf16_t*)dqkv, S, H, D, sl2, sc);
    }
    return hipGetLastError();
  }
  ProfScope ps("attn_bwd_generic", 8.0 * B * (double)S * S * D, 0, st);
  if (dtype == kBF16)
    return bwd_simple((const bf16_t*)qkv, (const bf16_t*)dO, lse, delta, (bf16_t*)dqkv, B, S, H, D, hd, st);
  return bwd_simple((const float*)qkv, (const float*)dO, lse, delta, (float*)dqkv, B, S, H, D, hd, st);
}

}  // namespace sr
