// GEMMs of the block (QKV, output projection, MLP; forward, dX and dW).
//
//   C[m, n] = sum_k A(m, k) * B(n, k)
//
// A(m,k) is either "k-major" (A[m*lda + k]) or "m-major" (A[k*lda + m]); B(n,k)
// likewise.  Forward X W^T is k-major x k-major; dX = dY W is k-major x n-major;
// dW = dY^T X is m-major x n-major (the reduction runs over tokens).
//
// gemm_mfma: bf16 operands, fp32 accumulation on gfx950 matrix cores
// (v_mfma_f32_32x32x16_bf16).  Workgroup tile 128 x 128 x 64, four waves in a
// 2 x 2 arrangement, each wave 64 x 64 = 2 x 2 MFMA tiles.  Operand tiles are
// staged in LDS in k-contiguous rows with an XOR swizzle of the 16-byte chunks;
// k-major operands go global -> LDS directly, m-major ones are transposed in
// registers (4 x 8 blocks) on the way in.  The next k-tile is in flight while the
// current one is consumed.
// Global loads go through buffer resources, so rows past the end of an operand
// read as zero: ragged token counts need no predicates in the main loop.
//
// gemm_simple: any element type, generic strides, fp32 FMA; used by the fp32
// storage mode and for the tiny adaLN modulation products.
//
// Epilogues (per element, fp32 value v = accumulator):
//   EPI_BIAS_ACT  out_act = Ta(v + bias)                           (QKV)
//   EPI_RESID     t = v + bias; [adaLN: a_save = Ta(t); t *= gate_b]
//                 out_f32 = resid + t; [out_st = T(out_f32)]       (O-proj, FC2)
//   EPI_GELU      z = v + bias; out_act = Ta(z); out_act2 = Ta(GELU(z))   (FC1)
//   EPI_DGELU     out_act = Ta(v * GELU'(z_in))                     (FC2 dX)
//   EPI_ACT       out_act = Ta(v)                                   (O-proj dX)
//   EPI_F32       out_f32[split] = v                                (dX for LN, dW partials)
//   EPI_F32_ACC   out_f32 += v                                      (dcond over blocks)
//   EPI_BIAS_F32  out_f32 = v + bias                                (adaLN modulation vectors)
//   EPI_DO        out_act = Ta(v); delta = per-head row sums of Ta(v) * O (attention backward)
//   EPI_DW        dW = v, db = row sums of A (weight and bias gradients); with split-K each
//                 split writes a partial plane and reduce_splits_kernel sums the planes in
//                 split order, so the result does not depend on scheduling.
#include "common.h"
#include "sr_internal.h"

namespace sr {

// GELU(z) = z Phi(z) and GELU'(z) = Phi(z) + z phi(z) with the standard normal CDF Phi and
// density phi (exact GELU, not the tanh form).  Phi comes from erfc in the Chebyshev-fitted form
// of Press et al. (Numerical Recipes, Sec. 6.2): with x = |z|/sqrt(2) and t = 1/(1 + x/2),
// erfc(x) = t exp(-x^2 + q(t)); here q is a degree-9 least-squares fit of log2(erfc(x) e^{x^2} / t)
// on t in (0, 1] (coefficients of our own fit, relative error of erfc <= 1.1e-7 for all x >= 0).
// Branch-free, one reciprocal and one exp2; the tails have relative, not absolute, accuracy.
SR_DEV float half_erfc_of(float z, float zz) {   // 0.5 erfc(|z|/sqrt(2)), zz = z*z
  const float t = __builtin_amdgcn_rcpf(fmaf(fabsf(z), 0.35355339059327376f, 1.0f));
  float q = 0.24651731550693512f;
  q = fmaf(q, t, -1.1861149072647095f);
  q = fmaf(q, t, 2.147474527359009f);
  q = fmaf(q, t, -1.6377531290054321f);
  q = fmaf(q, t, 0.40232160687446594f);
  q = fmaf(q, t, -0.2687568664550781f);
  q = fmaf(q, t, 0.13963006436824799f);
  q = fmaf(q, t, 0.5397006273269653f);
  q = fmaf(q, t, 1.4427292346954346f);
  q = fmaf(q, t, -2.8257482051849365f);   // constant term minus 1: the factor 1/2
  return t * __builtin_amdgcn_exp2f(fmaf(zz, -0.72134752044448170f, q));
}
SR_DEV float norm_cdf(float z, float zz) {
  const float h = half_erfc_of(z, zz);
  return z >= 0.f ? 1.0f - h : h;
}
SR_DEV float gelu_f(float z) { return z * norm_cdf(z, z * z); }
SR_DEV float gelu_grad_f(float z) {
  const float zz = z * z;
  // phi(z) = 2^(-z^2 log2(e)/2 - log2(sqrt(2 pi)))
  return norm_cdf(z, zz) + z * __builtin_amdgcn_exp2f(fmaf(zz, -0.72134752044448170f, -1.3257480647361593f));
}

template <int EPI, typename T, typename Ta>
SR_DEV void epilogue(const EpiArgs& e, int m, int n, float v) {
  const size_t o = (size_t)m * e.ldo + n;
  if constexpr (EPI == EPI_BIAS_ACT) {
    ((Ta*)e.out_act)[o] = from_f32<Ta>(v + to_f32<T>(((const T*)e.bias)[n]));
  } else if constexpr (EPI == EPI_RESID) {
    float t = v + to_f32<T>(((const T*)e.bias)[n]);
    if (e.gate) {
      ((Ta*)e.a_save)[o] = from_f32<Ta>(t);
      t *= e.gate[(size_t)(m / e.S) * e.gate_stride + n];
    }
    const float r = e.resid[o] + t;
    if (e.out_f32) e.out_f32[o] = r;
    if (e.out_st) ((T*)e.out_st)[o] = from_f32<T>(r);
  } else if constexpr (EPI == EPI_GELU) {
    const float z = v + to_f32<T>(((const T*)e.bias)[n]);
    ((Ta*)e.out_act)[o] = from_f32<Ta>(z);
    ((Ta*)e.out_act2)[o] = from_f32<Ta>(gelu_f(z));
  } else if constexpr (EPI == EPI_DGELU) {
    const float z = to_f32<Ta>(((const Ta*)e.z_in)[o]);
    ((Ta*)e.out_act)[o] = from_f32<Ta>(v * gelu_grad_f(z));
  } else if constexpr (EPI == EPI_ACT) {
    ((Ta*)e.out_act)[o] = from_f32<Ta>(v);
  } else if constexpr (EPI == EPI_F32) {
    e.out_f32[(size_t)blockIdx.z * e.split_stride + o] = v;
  } else if constexpr (EPI == EPI_F32_ACC) {
    e.out_f32[o] += v;
  } else if constexpr (EPI == EPI_BIAS_F32) {
    e.out_f32[o] = v + to_f32<T>(((const T*)e.bias)[n]);
  }
}

// ============================================================================ MFMA kernel

constexpr int GK = 64;
// s_waitcnt immediates (vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
constexpr int kLgkm0 = 0xC07F;   // LDS / scalar-memory counter at zero, the others untouched

// Operand tiles sit in LDS as rows of 64 bf16 (eight 16-byte chunks), unpadded; chunk c
// of row r is stored at chunk position c ^ ((r ^ (r >> 3)) & 7).  With it, the 16-byte
// fragment reads of eight consecutive rows, the k-major tile stores (eight chunks of a
// row) and the transposed 8-byte stores (eight rows 8 apart) all hit distinct banks.
SR_DEV int lds_off(int row, int chunk) { return row * GK + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 3); }

// Register staging of one R x 64 operand tile (R/32 16-byte vectors per thread).
template <int R>
struct TileRegs {
  i32x4 v[R / 32 > 4 ? R / 32 : 4];   // k-major: R/32 vectors; r-major: 4 per task
};

// k-major operand: rows r0.., k columns k0..k0+63 of X[r*ld + k].
template <int R>
SR_DEV void load_kmajor(TileRegs<R>& t, __amdgpu_buffer_rsrc_t rs, int r0, int k0, int ld) {
#pragma unroll
  for (int i = 0; i < R / 32; ++i) {
    const int c = threadIdx.x + 256 * i;
    const int row = c >> 3, kc = c & 7;
    const uint32_t off = ((uint32_t)(r0 + row) * (uint32_t)ld + (uint32_t)(k0 + kc * 8)) * 2u;
    t.v[i] = buf_load16(rs, off);
  }
}
template <int R>
SR_DEV void store_kmajor(const TileRegs<R>& t, bf16_t* lds) {
#pragma unroll
  for (int i = 0; i < R / 32; ++i) {
    const int c = threadIdx.x + 256 * i;
    *reinterpret_cast<i32x4*>(lds + lds_off(c >> 3, c & 7)) = t.v[i];
  }
}

// k-major operand straight from global memory into LDS (buffer_load ... lds, 16 bytes per
// lane): each wave fills whole 1 KB blocks (eight 128-byte rows), lane l landing at byte 16l
// of its block, so lane l fetches the logical chunk that the swizzle places at physical
// chunk l % 8 of row l / 8.  No VGPRs and no LDS-store instructions are involved.
template <int R>
SR_DEV void load_kmajor_direct(__amdgpu_buffer_rsrc_t rs, bf16_t* lds, int r0, int k0, int ld) {
  constexpr int BPW = R / 32;   // 1 KB blocks per wave (four waves)
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int i = 0; i < BPW; ++i) {
    const int blk = wid * BPW + i;
    const int row = blk * 8 + (lane >> 3);
    const int chunk = (lane & 7) ^ ((row ^ (row >> 3)) & 7);
    const uint32_t off = ((uint32_t)(r0 + row) * (uint32_t)ld + (uint32_t)(k0 + chunk * 8)) * 2u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t*)(lds + blk * 512), 16, off, 0, 0, 0);
  }
}

// r-major operand: X[k*ld + r]; a task covers 4 consecutive k x 8 consecutive r and is
// transposed in registers into eight 4-element k runs (R/128 tasks per thread).
template <int R>
SR_DEV void load_rmajor(TileRegs<R>& t, __amdgpu_buffer_rsrc_t rs, int r0, int k0, int ld) {
  constexpr int NRC = R / 8;
#pragma unroll
  for (int p = 0; p < (R + 127) / 128; ++p) {
    const int task = threadIdx.x + 256 * p;
    if (R < 128 && task >= 2 * R) break;   // 2R tasks of 4 k x 8 r
    const int rc = task % NRC, kg = task / NRC;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t off = ((uint32_t)(k0 + kg * 4 + i) * (uint32_t)ld + (uint32_t)(r0 + rc * 8)) * 2u;
      t.v[p * 4 + i] = buf_load16(rs, off);
    }
  }
}
template <int R>
SR_DEV void store_rmajor(const TileRegs<R>& t, bf16_t* lds) {
  constexpr int NRC = R / 8;
#pragma unroll
  for (int p = 0; p < (R + 127) / 128; ++p) {
    const int task = threadIdx.x + 256 * p;
    if (R < 128 && task >= 2 * R) break;
    const int rc = task % NRC, kg = task / NRC;
    const uint16_t* e0 = reinterpret_cast<const uint16_t*>(&t.v[p * 4 + 0]);
    const uint16_t* e1 = reinterpret_cast<const uint16_t*>(&t.v[p * 4 + 1]);
    const uint16_t* e2 = reinterpret_cast<const uint16_t*>(&t.v[p * 4 + 2]);
    const uint16_t* e3 = reinterpret_cast<const uint16_t*>(&t.v[p * 4 + 3]);
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      i32x2 w;
      w[0] = (int)((uint32_t)e0[r] | ((uint32_t)e1[r] << 16));
      w[1] = (int)((uint32_t)e2[r] | ((uint32_t)e3[r] << 16));
      *reinterpret_cast<i32x2*>(lds + lds_off(rc * 8 + r, kg >> 1) + (kg & 1) * 4) = w;
    }
  }
}

// Vectorised epilogue on four consecutive columns n..n+3 of row m (inputs already loaded).
struct EpiIn {
  f32x4 resid;
  i32x2 z;     // four activation-type values (bf16) of the GELU pre-activation
  f32x4 zf;    // the same for fp32 activations (unused in the MFMA path)
};

template <int EPI>
SR_DEV void epi_load(const EpiArgs& e, int m, int n, EpiIn& in) {
  const size_t o = (size_t)m * e.ldo + n;
  if constexpr (EPI == EPI_RESID) in.resid = *reinterpret_cast<const f32x4*>(e.resid + o);
  if constexpr (EPI == EPI_DGELU) in.z = *reinterpret_cast<const i32x2*>((const bf16_t*)e.z_in + o);
  if constexpr (EPI == EPI_F32_ACC) in.resid = *reinterpret_cast<const f32x4*>(e.out_f32 + o);
  if constexpr (EPI == EPI_DO) in.z = *reinterpret_cast<const i32x2*>((const bf16_t*)e.o_in + o);
}

SR_DEV i32x2 pack4(f32x4 v) {
  i32x2 w;
  w[0] = (int)f2bf2(v[0], v[1]);
  w[1] = (int)f2bf2(v[2], v[3]);
  return w;
}

// Returns the EPI_DO partial sum of this chunk (0 otherwise).
template <int EPI>
SR_DEV float epi_store(const EpiArgs& e, int m, int n, f32x4 v, const EpiIn& in) {
  const size_t o = (size_t)m * e.ldo + n;
  f32x4 b = {0.f, 0.f, 0.f, 0.f};
  if constexpr (EPI == EPI_BIAS_ACT || EPI == EPI_RESID || EPI == EPI_GELU || EPI == EPI_BIAS_F32) {
    const i32x2 bw = *reinterpret_cast<const i32x2*>((const bf16_t*)e.bias + n);
    const bf16_t* be = reinterpret_cast<const bf16_t*>(&bw);
#pragma unroll
    for (int q = 0; q < 4; ++q) b[q] = bf2f(be[q]);
  }
  if constexpr (EPI == EPI_BIAS_ACT) {
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = pack4(v + b);
  } else if constexpr (EPI == EPI_RESID) {
    f32x4 t = v + b;
    if (e.gate) {
      *reinterpret_cast<i32x2*>((bf16_t*)e.a_save + o) = pack4(t);
      t *= *reinterpret_cast<const f32x4*>(e.gate + (size_t)(m / e.S) * e.gate_stride + n);
    }
    const f32x4 r = in.resid + t;
    if (e.out_f32) *reinterpret_cast<f32x4*>(e.out_f32 + o) = r;
    if (e.out_st) *reinterpret_cast<i32x2*>((bf16_t*)e.out_st + o) = pack4(r);
  } else if constexpr (EPI == EPI_GELU) {
    const f32x4 z = v + b;
    f32x4 gz;
#pragma unroll
    for (int q = 0; q < 4; ++q) gz[q] = gelu_f(z[q]);
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = pack4(z);
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act2 + o) = pack4(gz);
  } else if constexpr (EPI == EPI_DGELU) {
    const bf16_t* ze = reinterpret_cast<const bf16_t*>(&in.z);
    f32x4 d;
#pragma unroll
    for (int q = 0; q < 4; ++q) d[q] = v[q] * gelu_grad_f(bf2f(ze[q]));
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = pack4(d);
  } else if constexpr (EPI == EPI_ACT) {
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = pack4(v);
  } else if constexpr (EPI == EPI_F32) {
    *reinterpret_cast<f32x4*>(e.out_f32 + (size_t)blockIdx.z * e.split_stride + o) = v;
  } else if constexpr (EPI == EPI_F32_ACC) {
    *reinterpret_cast<f32x4*>(e.out_f32 + o) = in.resid + v;
  } else if constexpr (EPI == EPI_BIAS_F32) {
    *reinterpret_cast<f32x4*>(e.out_f32 + o) = v + b;
  } else if constexpr (EPI == EPI_DW) {
    float* out = gridDim.z == 1 ? e.out_f32 : e.part + (size_t)blockIdx.z * e.split_stride;
    *reinterpret_cast<f32x4*>(out + o) = v;
  } else if constexpr (EPI == EPI_DO) {
    const i32x2 w = pack4(v);
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = w;
    const bf16_t* de = reinterpret_cast<const bf16_t*>(&w);
    const bf16_t* oe = reinterpret_cast<const bf16_t*>(&in.z);
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) s += bf2f(de[q]) * bf2f(oe[q]);
    return s;
  }
  return 0.f;
}

// BM x BN workgroup tile, four waves in 2 x 2, each (BM/2) x (BN/2), i.e. MI x NJ MFMA tiles
// of 32 x 32 (MI = BM/64, NJ = BN/64).  A wave reads (MI + NJ) KB of fragments from LDS per
// MI * NJ MFMAs, so the big tiles (one workgroup per CU, accumulators in AGPRs) need half the
// LDS bandwidth of 128 x 128 per MFMA; 128 x 128 and 64 x 128 keep two workgroups per CU and
// enough tiles for narrow outputs.
template <int BM, int BN, bool AK, bool BK, int EPI, typename T, typename Ta>
__global__ __launch_bounds__(256, BM * BN >= 256 * 128 ? 1 : 2) void gemm_mfma_kernel(
    const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bm, int M, int N, int Kd, int lda, int ldb,
    uint32_t a_bytes, uint32_t b_bytes, int k_per_split, EpiArgs ep) {
  constexpr int MI = BM / 64 > 0 ? BM / 64 : 1;
  constexpr int NJ = BN / 64;
  static_assert(BM == 64 || BM == 128 || BM == 256, "tile height");
  static_assert(BN == 128 || BN == 256, "tile width");
  constexpr int GN = BN;
  constexpr int STAGE = (BM + BN) * GK;   // bf16 elements of one LDS stage (A tile then B tile)
  constexpr int EPI_LD = BN + 8;          // fp32 row stride of the epilogue staging tile
  constexpr int PR = BN == 256 ? (BM < 64 ? BM : 64) : (BM < 128 ? BM : 128);   // rows per pass
  constexpr int EPI_BYTES = PR * EPI_LD * 4;
  constexpr int SMEM = EPI_BYTES > 2 * STAGE * 2 ? EPI_BYTES : 2 * STAGE * 2;
  // two operand stages (the next k-tile is written into one while the other is consumed);
  // the same memory stages the fp32 result, 128 rows at a time, for the epilogue
  __shared__ __attribute__((aligned(16))) char smem_raw[SMEM];
  bf16_t* smem = reinterpret_cast<bf16_t*>(smem_raw);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int wm = wid >> 1, wn = wid & 1;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * GN;
  const int kbeg = blockIdx.z * k_per_split;
  const int kend = min(Kd, kbeg + k_per_split);
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(Bm, b_bytes);

  f32x16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // k-major operands go global -> LDS directly; r-major ones through registers (transposed)
  TileRegs<BM> ta;
  TileRegs<GN> tb;
  auto gload = [&](int k0, int s) {
    bf16_t* st = smem + s * STAGE;
    if constexpr (AK) load_kmajor_direct<BM>(ra, st, m0, k0, lda); else load_rmajor<BM>(ta, ra, m0, k0, lda);
    if constexpr (BK) load_kmajor_direct<GN>(rb, st + BM * GK, n0, k0, ldb); else load_rmajor<GN>(tb, rb, n0, k0, ldb);
  };
  auto lstore = [&](int s) {
    bf16_t* st = smem + s * STAGE;
    if constexpr (!AK) store_rmajor<BM>(ta, st);
    if constexpr (!BK) store_rmajor<GN>(tb, st + BM * GK);
  };

  // EPI_DW: the first column of tiles also sums its A rows (bias gradient)
  constexpr int TPR = 256 / BM;   // threads per A row for those sums
  const bool do_db = EPI == EPI_DW && ep.db_out != nullptr && blockIdx.x == 0;
  float dbacc = 0.f;

  const int h = lane >> 5;
  // LDS offsets of this lane's fragment rows (the stage and k-step are added per use)
  int aoff[MI], boff[NJ], asw[MI], bsw[NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int row = wm * (BM / 2) + i * 32 + (lane & 31);
    aoff[i] = row * GK;
    asw[i] = (row ^ (row >> 3)) & 7;
  }
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int row = wn * (BN / 2) + j * 32 + (lane & 31);
    boff[j] = BM * GK + row * GK;
    bsw[j] = (row ^ (row >> 3)) & 7;
  }

  // Software pipeline (two LDS stages, two fragment buffers).  Per k-tile t, k-steps
  // 0..KS-2 each read the next step's fragments and then issue this step's MFMAs; the
  // workgroup barrier sits before the last k-step, after which tile t's stage is free for
  // tile t+2's loads and tile t+1's first fragments are read while the last step's MFMAs
  // run.  sched_barrier keeps the compiler from sinking the reads to their first use.
  constexpr int KS = GK / 16;
  const int ntile = kbeg < kend ? (kend - kbeg + GK - 1) / GK : 0;
  bf16x8 fa[2][MI], fb[2][NJ];
  auto read_frags = [&](int s, int ks, int buf) {
    const bf16_t* St = smem + s * STAGE;
#pragma unroll
    for (int i = 0; i < MI; ++i)
      fa[buf][i] = *reinterpret_cast<const bf16x8*>(St + aoff[i] + (((2 * ks + h) ^ asw[i]) << 3));
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      fb[buf][j] = *reinterpret_cast<const bf16x8*>(St + boff[j] + (((2 * ks + h) ^ bsw[j]) << 3));
  };
  auto mfmas = [&](int buf) {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][i], fb[buf][j], acc[i][j], 0, 0, 0);
  };

  if (ntile > 0) {
    gload(kbeg, 0);
    lstore(0);
  }
  __builtin_amdgcn_s_waitcnt(0);   // direct LDS loads are counted by vmcnt
  __syncthreads();
  if (ntile > 0) read_frags(0, 0, 0);
  if (ntile > 1) gload(kbeg + GK, 1);
  __builtin_amdgcn_s_waitcnt(kLgkm0);
  for (int it = 0; it < ntile; ++it) {
    const int cur = it & 1;
    const bool more = it + 1 < ntile;
    if (do_db) {
      const bf16_t* St = smem + cur * STAGE;
      const int row = threadIdx.x / TPR;
#pragma unroll
      for (int q = 0; q < 8 / TPR; ++q) {
        i32x4 v = *reinterpret_cast<const i32x4*>(St + lds_off(row, (threadIdx.x % TPR) * (8 / TPR) + q));
        const bf16_t* e = reinterpret_cast<const bf16_t*>(&v);
#pragma unroll
        for (int j = 0; j < 8; ++j) dbacc += bf2f(e[j]);
      }
    }
#pragma unroll
    for (int ks = 0; ks < KS - 1; ++ks) {
      read_frags(cur, ks + 1, (ks + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
      mfmas(ks & 1);
      __builtin_amdgcn_sched_barrier(0);
    }
    if (more) lstore(cur ^ 1);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of tile it+1 have landed
    __syncthreads();                 // ... and every wave's; tile it's stage is no longer read
    if (it + 2 < ntile) gload(kbeg + (it + 2) * GK, cur);
    if (more) read_frags(cur ^ 1, 0, KS & 1);
    __builtin_amdgcn_sched_barrier(0);
    mfmas((KS - 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
    // the next tile's first fragments were requested a whole k-step ago: settle them here
    // so that the top of the loop does not wait for the reads it issues itself
    __builtin_amdgcn_s_waitcnt(kLgkm0);
  }

  if constexpr (EPI == EPI_DW) {
#pragma unroll
    for (int o = 1; o < TPR; o <<= 1) dbacc += __shfl_xor(dbacc, o, 64);
    const int dbrow = m0 + (int)threadIdx.x / TPR;
    if (do_db && (threadIdx.x % TPR) == 0 && dbrow < M) {
      if (gridDim.z == 1) ep.db_out[dbrow] = dbacc;
      else ep.dbpart[(size_t)blockIdx.z * M + dbrow] = dbacc;
    }
  }

  // epilogue, PR rows per pass: stage the fp32 result (register r of a 32x32 MFMA tile
  // holds row 8*(r/4) + 4*(lane/32) + r%4, column lane%32), then 4-column chunks per thread
  constexpr int CPR = BN / 4;                   // 4-column chunks per row
  constexpr int NB = PR * CPR / (256 * 8);      // batches of 8 chunks per thread in a pass
  static_assert(NB >= 1 && NB * 256 * 8 == PR * CPR, "epilogue pass shape");
  float* stage = reinterpret_cast<float*>(smem_raw);
#pragma unroll
  for (int half = 0; half < BM / PR; ++half) {
    if (half) __syncthreads();
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm * (BM / 2) + i * 32 + 8 * (r >> 2) + 4 * h + (r & 3) - half * PR;
          const int col = wn * (BN / 2) + j * 32 + (lane & 31);
          if (row >= 0 && row < PR) stage[row * EPI_LD + col] = acc[i][j][r];
        }
    __syncthreads();
#pragma unroll
    for (int bch = 0; bch < NB; ++bch) {
      EpiIn in[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int c = threadIdx.x + 256 * (bch * 8 + q);
        const int m = m0 + half * PR + c / CPR, n = n0 + (c % CPR) * 4;
        if (m < M && n < N) epi_load<EPI>(ep, m, n, in[q]);
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int c = threadIdx.x + 256 * (bch * 8 + q);
        const int row = c / CPR, c4 = (c % CPR) * 4;
        const int m = m0 + half * PR + row, n = n0 + c4;
        float part = 0.f;
        if (m < M && n < N)
          part = epi_store<EPI>(ep, m, n, *reinterpret_cast<const f32x4*>(stage + row * EPI_LD + c4), in[q]);
        if constexpr (EPI == EPI_DO) {
          // the 16 lanes (tid % 16) of one head's 64 columns: butterfly within the group
#pragma unroll
          for (int o = 8; o >= 1; o >>= 1) part += __shfl_xor(part, o, 64);
          if ((threadIdx.x & 15) == 0 && m < M && n < N)
            ep.delta[((size_t)(m / ep.S) * ep.H + (n >> 6)) * ep.S + (m % ep.S)] = part;
        }
      }
    }
  }
}

// Sum of split-K partial planes, in split order: out[i] = sum_z part[z * n + i] (float4 lanes),
// and likewise for the bias-gradient partials.
__global__ __launch_bounds__(256) void reduce_splits_kernel(const float* __restrict__ part, int splits, size_t n4,
                                                            float* __restrict__ out, const float* __restrict__ dbpart,
                                                            int nb, float* __restrict__ dbout) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n4) {
    const f32x4* p = reinterpret_cast<const f32x4*>(part);
    f32x4 s = p[i];
    for (int z = 1; z < splits; ++z) s += p[(size_t)z * n4 + i];
    reinterpret_cast<f32x4*>(out)[i] = s;
  } else if (dbout && i - n4 < (size_t)nb) {
    const size_t c = i - n4;
    float s = dbpart[c];
    for (int z = 1; z < splits; ++z) s += dbpart[(size_t)z * nb + c];
    dbout[c] = s;
  }
}

hipError_t launch_reduce_splits(const float* part, int splits, size_t n, float* out, const float* dbpart, int nb,
                                float* dbout, hipStream_t st) {
  const size_t n4 = n / 4;
  const size_t total = n4 + (dbout ? nb : 0);
  hipLaunchKernelGGL(reduce_splits_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, part, splits, n4,
                     out, dbpart, nb, dbout);
  return hipGetLastError();
}

// ============================================================================ generic kernel

template <typename TA, typename TB, int EPI, typename T, typename Ta>
__global__ __launch_bounds__(256) void gemm_simple_kernel(const TA* __restrict__ A, const TB* __restrict__ Bm, int M,
                                                          int N, int Kd, long long a_sm, long long a_sk,
                                                          long long b_sn, long long b_sk, EpiArgs ep) {
  __shared__ float As[16][65];
  __shared__ float Bs[16][65];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  const bool do_db = EPI == EPI_DW && ep.db_out != nullptr && blockIdx.x == 0;
  float dbacc = 0.f;
  for (int k0 = 0; k0 < Kd; k0 += 16) {
    for (int t = threadIdx.x; t < 64 * 16; t += 256) {
      const int kk = t >> 6, r = t & 63;
      const int m = m0 + r, n = n0 + r, k = k0 + kk;
      As[kk][r] = (m < M && k < Kd) ? to_f32<TA>(A[m * a_sm + k * a_sk]) : 0.f;
      Bs[kk][r] = (n < N && k < Kd) ? to_f32<TB>(Bm[n * b_sn + k * b_sk]) : 0.f;
    }
    __syncthreads();
    if (do_db && threadIdx.x < 64)
      for (int kk = 0; kk < 16; ++kk) dbacc += As[kk][threadIdx.x];
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }
  if (do_db && threadIdx.x < 64 && m0 + (int)threadIdx.x < M) ep.db_out[m0 + threadIdx.x] = dbacc;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
      if (m < M && n < N) {
        if constexpr (EPI == EPI_DW) ep.out_f32[(size_t)m * ep.ldo + n] = acc[i][j];
        else epilogue<EPI, T, Ta>(ep, m, n, acc[i][j]);
      }
    }
}

// ============================================================================ dispatch

template <int BM, int BN, int EPI, typename T, typename Ta>
static hipError_t run_mfma_tile(const GemmDesc& g, const EpiArgs& ep, hipStream_t st) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, g.splits);
  const int kps = g.splits > 1 ? g.k_per_split : g.K;
#define SR_GEMM_L(AK, BK)                                                                                         \
  hipLaunchKernelGGL((gemm_mfma_kernel<BM, BN, AK, BK, EPI, T, Ta>), grid, dim3(256), 0, st, (const bf16_t*)g.A,   \
                     (const bf16_t*)g.B, g.M, g.N, g.K, (int)g.lda, (int)g.ldb, (uint32_t)g.a_bytes,              \
                     (uint32_t)g.b_bytes, kps, ep)
  if (g.a_kmajor && g.b_kmajor) SR_GEMM_L(true, true);
  else if (g.a_kmajor && !g.b_kmajor) SR_GEMM_L(true, false);
  else if (!g.a_kmajor && !g.b_kmajor) SR_GEMM_L(false, false);
  else SR_GEMM_L(false, true);
#undef SR_GEMM_L
  return hipGetLastError();
}

// Tile shape: 128 x 128, or 64 x 128 when 128 x 128 tiles would leave fewer than two
// workgroups per CU.
template <int EPI, typename T, typename Ta>
static hipError_t run_mfma(const GemmDesc& g, const EpiArgs& ep, hipStream_t st) {
  const long tiles128 = (long)((g.N + 127) / 128) * ((g.M + 127) / 128) * g.splits;
#ifdef SR_GEMM_FORCE_TILE
  // standalone benchmarks: 0 = 64x128, 1 = 128x128, 2 = 256x128, 3 = 128x256, 4 = 256x256
  switch (SR_GEMM_FORCE_TILE) {
    case 0: return run_mfma_tile<64, 128, EPI, T, Ta>(g, ep, st);
    case 1: return run_mfma_tile<128, 128, EPI, T, Ta>(g, ep, st);
    case 2: return run_mfma_tile<256, 128, EPI, T, Ta>(g, ep, st);
    case 3: return run_mfma_tile<128, 256, EPI, T, Ta>(g, ep, st);
    default: return run_mfma_tile<256, 256, EPI, T, Ta>(g, ep, st);
  }
#endif
  if (tiles128 < 512) return run_mfma_tile<64, 128, EPI, T, Ta>(g, ep, st);
  return run_mfma_tile<128, 128, EPI, T, Ta>(g, ep, st);
}

template <int EPI, typename T, typename Ta, typename TA, typename TB>
static hipError_t run_simple(const GemmDesc& g, const EpiArgs& ep, hipStream_t st) {
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, 1);
  const long long a_sm = g.a_kmajor ? g.lda : 1, a_sk = g.a_kmajor ? 1 : g.lda;
  const long long b_sn = g.b_kmajor ? g.ldb : 1, b_sk = g.b_kmajor ? 1 : g.ldb;
  hipLaunchKernelGGL((gemm_simple_kernel<TA, TB, EPI, T, Ta>), grid, dim3(256), 0, st, (const TA*)g.A,
                     (const TB*)g.B, g.M, g.N, g.K, a_sm, a_sk, b_sn, b_sk, ep);
  return hipGetLastError();
}

template <int EPI>
static hipError_t dispatch(const GemmDesc& g, const EpiArgs& ep, hipStream_t st) {
  if (g.use_mfma) return run_mfma<EPI, bf16_t, bf16_t>(g, ep, st);
  // simple path: element types of A and B, T/Ta = storage / activation type
  if (g.dtype == kBF16) {
    if (g.a_type == kBF16 && g.b_type == kBF16) return run_simple<EPI, bf16_t, bf16_t, bf16_t, bf16_t>(g, ep, st);
    if (g.a_type == kF32 && g.b_type == kBF16) return run_simple<EPI, bf16_t, bf16_t, float, bf16_t>(g, ep, st);
    if (g.a_type == kBF16 && g.b_type == kF32) return run_simple<EPI, bf16_t, bf16_t, bf16_t, float>(g, ep, st);
    return run_simple<EPI, bf16_t, bf16_t, float, float>(g, ep, st);
  }
  return run_simple<EPI, float, float, float, float>(g, ep, st);
}

hipError_t launch_gemm(const GemmDesc& g, int epi, const EpiArgs& ep, hipStream_t st) {
  switch (epi) {
    case EPI_BIAS_ACT: return dispatch<EPI_BIAS_ACT>(g, ep, st);
    case EPI_RESID: return dispatch<EPI_RESID>(g, ep, st);
    case EPI_GELU: return dispatch<EPI_GELU>(g, ep, st);
    case EPI_DGELU: return dispatch<EPI_DGELU>(g, ep, st);
    case EPI_ACT: return dispatch<EPI_ACT>(g, ep, st);
    case EPI_F32: return dispatch<EPI_F32>(g, ep, st);
    case EPI_F32_ACC: return dispatch<EPI_F32_ACC>(g, ep, st);
    case EPI_BIAS_F32: return dispatch<EPI_BIAS_F32>(g, ep, st);
    case EPI_DW: return dispatch<EPI_DW>(g, ep, st);
    case EPI_DO: return g.use_mfma ? run_mfma<EPI_DO, bf16_t, bf16_t>(g, ep, st) : hipErrorInvalidValue;
  }
  return hipErrorInvalidValue;
}

}  // namespace sr
