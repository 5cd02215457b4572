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
//   EPI_GELU      z = Ta(v + bias); out_act = z; out_act2 = Ta(GELU(z))    (FC1)
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
// erfc(x) = t exp(-x^2 + q(t)); here q is a least-squares polynomial fit of
// log2(erfc(x) e^{x^2} / t) on t in (0, 1] (coefficients of our own fits), of degree 9 for fp32
// activations and 5 for bf16 ones.  Evaluated in fp32 the relative error of erfc is, at degree 9,
// below 2e-7 for x <= 4 and grows to 1.4e-5 near x = 8, where the rounding of the exponent
// argument (about -92) dominates; at degree 5 it stays below 4.8e-5 for x <= 8.  bf16 outputs
// round at 2e-3, forty times coarser, and the fp32 mode's gradients need the degree-9 fit.
// Branch-free, one reciprocal and one exp2; the tails have relative, not absolute, accuracy.
template <int DEG>
SR_DEV float half_erfc_of(float z, float zz) {   // 0.5 erfc(|z|/sqrt(2)), zz = z*z
  static_assert(DEG == 5 || DEG == 9, "fit degree");
  const float t = __builtin_amdgcn_rcpf(fmaf(fabsf(z), 0.35355339059327376f, 1.0f));
  float q;
  if constexpr (DEG == 9) {
    q = 0.24651731550693512f;
    q = fmaf(q, t, -1.1861149072647095f);
    q = fmaf(q, t, 2.147474527359009f);
    q = fmaf(q, t, -1.6377531290054321f);
    q = fmaf(q, t, 0.40232160687446594f);
    q = fmaf(q, t, -0.2687568664550781f);
    q = fmaf(q, t, 0.13963006436824799f);
    q = fmaf(q, t, 0.5397006273269653f);
    q = fmaf(q, t, 1.4427292346954346f);
    q = fmaf(q, t, -2.8257482051849365f);   // constant term minus 1: the factor 1/2
  } else {
    q = 0.278960645198822f;
    q = fmaf(q, t, -0.8764582872390747f);
    q = fmaf(q, t, 0.52732914686203f);
    q = fmaf(q, t, 0.44432464241981506f);
    q = fmaf(q, t, 1.451727271080017f);
    q = fmaf(q, t, -2.82594895362854f);     // constant term minus 1: the factor 1/2
  }
  return t * __builtin_amdgcn_exp2f(fmaf(zz, -0.72134752044448170f, q));
}
// fit degree for an activation storage type
template <typename Ta>
constexpr int gelu_deg() {
  return sizeof(Ta) == 2 ? 5 : 9;
}
template <int DEG>
SR_DEV float norm_cdf(float z, float zz) {
  const float h = half_erfc_of<DEG>(z, zz);
  return z >= 0.f ? 1.0f - h : h;
}
template <int DEG>
SR_DEV float gelu_f(float z) {
  return z * norm_cdf<DEG>(z, z * z);
}
template <int DEG>
SR_DEV float gelu_grad_f(float z) {
  const float zz = z * z;
  // phi(z) = 2^(-z^2 log2(e)/2 - log2(sqrt(2 pi)))
  return norm_cdf<DEG>(z, zz) + z * __builtin_amdgcn_exp2f(fmaf(zz, -0.72134752044448170f, -1.3257480647361593f));
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
    if (e.sc_x) {
      const int b = m / e.S, s = m - b * e.S;
      const int i = e.sc_idx[(e.sc_shared ? 0 : b) * e.S + s];
      T* xp = (T*)e.sc_x + ((size_t)b * e.sc_L + i) * e.ldo + n;
      const float x0 = to_f32<T>(*xp);
      *xp = from_f32<T>(__fadd_rn(x0, __fsub_rn(to_f32<T>(from_f32<T>(r)), x0)));
    }
  } else if constexpr (EPI == EPI_GELU) {
    const Ta z = from_f32<Ta>(v + to_f32<T>(((const T*)e.bias)[n]));
    ((Ta*)e.out_act)[o] = z;
    ((Ta*)e.out_act2)[o] = from_f32<Ta>(gelu_f<gelu_deg<Ta>()>(to_f32<Ta>(z)));   // of the stored z (recomputed bit for bit)
  } else if constexpr (EPI == EPI_DGELU) {
    const float z = to_f32<Ta>(((const Ta*)e.z_in)[o]);
    ((Ta*)e.out_act)[o] = from_f32<Ta>(v * gelu_grad_f<gelu_deg<Ta>()>(z));
  } else if constexpr (EPI == EPI_ACT) {
    ((Ta*)e.out_act)[o] = from_f32<Ta>(v);
  } else if constexpr (EPI == EPI_F32) {
    e.out_f32[o] = v;
  } else if constexpr (EPI == EPI_F32_ACC) {
    e.out_f32[o] += v;
  } else if constexpr (EPI == EPI_BIAS_F32) {
    e.out_f32[o] = v + to_f32<T>(((const T*)e.bias)[n]);
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
SR_DEV f32x4 unpack4(i32x2 w) {
  f32x4 v;
  v[0] = __uint_as_float((uint32_t)w[0] << 16);
  v[1] = __uint_as_float((uint32_t)w[0] & 0xFFFF0000u);
  v[2] = __uint_as_float((uint32_t)w[1] << 16);
  v[3] = __uint_as_float((uint32_t)w[1] & 0xFFFF0000u);
  return v;
}

constexpr bool epi_has_bias(int epi) {
  return epi == EPI_BIAS_ACT || epi == EPI_RESID || epi == EPI_GELU || epi == EPI_BIAS_F32;
}

// Bias of the four columns n..n+3 (zero for epilogues without one).
template <int EPI>
SR_DEV f32x4 epi_bias(const EpiArgs& e, int n) {
  f32x4 b = {0.f, 0.f, 0.f, 0.f};
  if constexpr (epi_has_bias(EPI)) {
    const i32x2 bw = *reinterpret_cast<const i32x2*>((const bf16_t*)e.bias + n);
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      b[2 * q] = __uint_as_float((uint32_t)bw[q] << 16);
      b[2 * q + 1] = __uint_as_float((uint32_t)bw[q] & 0xFFFF0000u);
    }
  }
  return b;
}

// Returns the EPI_DO partial sum of this chunk (0 otherwise).  b: the columns' bias (epi_bias).
template <int EPI>
SR_DEV float epi_store(const EpiArgs& e, int m, int n, f32x4 v, const EpiIn& in, f32x4 b) {
  const size_t o = (size_t)m * e.ldo + n;
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
    if (e.sc_x) {
      const int b = m / e.S, s = m - b * e.S;
      const int i = e.sc_idx[(e.sc_shared ? 0 : b) * e.S + s];
      bf16_t* xp = (bf16_t*)e.sc_x + ((size_t)b * e.sc_L + i) * e.ldo + n;
      const f32x4 x0 = unpack4(*reinterpret_cast<const i32x2*>(xp));
      const f32x4 h = unpack4(pack4(r));
      f32x4 xn;
#pragma unroll
      for (int q = 0; q < 4; ++q) xn[q] = __fadd_rn(x0[q], __fsub_rn(h[q], x0[q]));
      *reinterpret_cast<i32x2*>(xp) = pack4(xn);
    }
  } else if constexpr (EPI == EPI_GELU) {
    // GELU of the stored (rounded) pre-activation, so the backward recomputes it bit for bit
    const i32x2 zb = pack4(v + b);
    const f32x4 z = unpack4(zb);
    f32x4 gz;
#pragma unroll
    for (int q = 0; q < 4; ++q) gz[q] = gelu_f<gelu_deg<bf16_t>()>(z[q]);
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = zb;
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act2 + o) = pack4(gz);
  } else if constexpr (EPI == EPI_DGELU) {
    const bf16_t* ze = reinterpret_cast<const bf16_t*>(&in.z);
    f32x4 d;
#pragma unroll
    for (int q = 0; q < 4; ++q) d[q] = v[q] * gelu_grad_f<gelu_deg<bf16_t>()>(bf2f(ze[q]));
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = pack4(d);
  } else if constexpr (EPI == EPI_ACT) {
    *reinterpret_cast<i32x2*>((bf16_t*)e.out_act + o) = pack4(v);
  } else if constexpr (EPI == EPI_F32) {
    *reinterpret_cast<f32x4*>(e.out_f32 + o) = v;
  } else if constexpr (EPI == EPI_F32_ACC) {
    *reinterpret_cast<f32x4*>(e.out_f32 + o) = in.resid + v;
  } else if constexpr (EPI == EPI_BIAS_F32) {
    *reinterpret_cast<f32x4*>(e.out_f32 + o) = v + b;
  } else if constexpr (EPI == EPI_DW) {
    *reinterpret_cast<f32x4*>(e.out_f32 + o) = v;   // the split's partial plane when split
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

// ============================================================================ MFMA kernel

constexpr int GK = 64;        // k extent of an operand tile
constexpr int KS = GK / 16;   // MFMA k-steps per tile

// LDS layouts of an operand tile (16-byte chunks of eight bf16 at XOR-swizzled positions):
//  k-major, R rows x 64 k: row r holds its 64 k values, chunk c at position c ^ kswz(r).  The
//    fragment reads (16 lanes: one chunk of 16 consecutive rows) hit distinct banks.
//  r-major, 64 k-rows x R: k-row k holds R consecutive r values, chunk c at c ^ rswz(k).
//    Fragments come from ds_read_b64_tr_b16; the four k-rows x 32 bytes that half a wave
//    touches per read sit in four different 64-byte bank groups.
// Both are filled by whole 1 KB blocks of contiguous LDS, so the fills are conflict-free.
SR_DEV int kswz(int r) { return (r ^ (r >> 3)) & 7; }
template <int R>
SR_DEV int rswz(int k) {
  return R >= 128 ? (k & 3) << 2 : ((k >> 1) & 1) << 2;
}

// One operand tile (R rows or r-columns, k0 .. k0+63) straight from global memory into LDS
// (buffer_load ... lds, 16 bytes per lane, no VGPRs): each wave fills whole 1 KB blocks and
// lane l lands at byte 16 l of its block, so it fetches the chunk the swizzle places there.
// Offsets at or past the operand's extent read as zero.  The lane's byte offsets for k0 = 0 are
// computed once; a tile adds one wave-uniform byte offset (k0 * 2 for k-major operands,
// k0 * ld * 2 for r-major ones), and the LDS block addresses are wave-uniform too, so a fill
// costs one vector add per load.
template <int R, bool KMAJ>
struct TileFill {
  static constexpr int BPW = R / 32;   // the tile is R/8 blocks of 1 KB, four waves
  uint32_t off[BPW];
  SR_DEV void init(int r0, int ld, int lane, int wid) {
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int blk = wid * BPW + i;
      if constexpr (KMAJ) {
        const int row = blk * 8 + (lane >> 3);
        const int c = (lane & 7) ^ kswz(row);
        off[i] = ((uint32_t)(r0 + row) * (uint32_t)ld + (uint32_t)(c * 8)) * 2u;
      } else {
        constexpr int CPR = R / 8, RPB = 64 / CPR;   // chunks per k-row, k-rows per block
        const int k = blk * RPB + lane / CPR;
        const int c = (lane % CPR) ^ rswz<R>(k);
        off[i] = ((uint32_t)k * (uint32_t)ld + (uint32_t)(r0 + c * 8)) * 2u;
      }
    }
  }
};

// Issue one tile's fills.  delta: the wave-uniform byte offset of k0, or 0x80000000 for a fill
// past the last k-tile, which keeps the count of loads in flight uniform: every offset then lies
// at or beyond 2 GiB, past every operand's extent, and reads zeros without a memory access.
// (It takes the offsets array: a function that takes the buffer resource together with the
// TileFill structure, member or not, fails in the host compilation pass, which then drops the
// kernels' launch stubs.)
template <int BPW>
SR_DEV void fill_issue(const uint32_t* off, __amdgpu_buffer_rsrc_t rs, bf16_t* lds, int wid, uint32_t delta) {
#pragma unroll
  for (int i = 0; i < BPW; ++i)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t*)(lds + (wid * BPW + i) * 512), 16, off[i] + delta, 0, 0,
                                             0);
}

// Workgroups are handed to the eight XCDs round-robin by linear id.  Renumber them so that each
// XCD owns a contiguous range of tiles, and walk tiles in groups of GM tile rows (column by
// column within a group), so the tiles that one XCD runs together share A rows and B columns in
// its L2.  Split-K index outermost.
constexpr int GM = 8;
SR_DEV void tile_coords(int bid, int nwg, int tiles_m, int tiles_n, int& tm, int& tn, int& split) {
  const int x = bid & 7, q = nwg >> 3, rem = nwg & 7;
  const int t = x * q + min(x, rem) + (bid >> 3);
  const int per = tiles_m * tiles_n;
  split = t / per;
  const int u = t - split * per;
  const int grp = u / (GM * tiles_n);
  const int first = grp * GM;
  const int gm = min(GM, tiles_m - first);
  const int v = u - first * tiles_n;
  tm = first + v % gm;
  tn = v / gm;
}


// Per-lane LDS byte addresses of one operand's fragments (stage 0, k-step 0 for r-major).
//  k-major: rows rb + 32 p + lane % 32 (p = 0, 1; rows 64 apart share the swizzle), one address
//    per k-step (the swizzle does not add).
//  r-major: r-columns rb + 32 i + ..., one address per i (k-steps and the second read of a
//    fragment are constant offsets: the swizzle depends on k % 4 only).
template <int R, bool KMAJ, int NI>
struct FragAddr {
  uint32_t a[KMAJ ? 2 : NI][KMAJ ? KS : 1];
  SR_DEV void init(uint32_t base, int rb, int lane) {
    const int h = lane >> 5;
    if constexpr (KMAJ) {
#pragma unroll
      for (int p = 0; p < (NI > 1 ? 2 : 1); ++p) {
        const int r = rb + 32 * p + (lane & 31);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) a[p][ks] = base + (uint32_t)(r * GK + (((2 * ks + h) ^ kswz(r)) << 3)) * 2u;
      }
    } else {
      const int g = lane >> 4, s = lane & 15;
      const int k1 = 8 * (g >> 1) + (s >> 2);
#pragma unroll
      for (int i = 0; i < NI; ++i) {
        const int col = rb + 32 * i + 16 * (g & 1) + 4 * (s & 3);
        a[i][0] = base + (uint32_t)(k1 * R + (((col >> 3) ^ rswz<R>(k1)) << 3) + (col & 7)) * 2u;
      }
    }
  }
  // fragment I at k-step KSV, byte offset OFF (stage and operand position): rows (or r-columns)
  // rb + 32 I + lane % 32, k = 16 KSV + 8 h .. + 7
  template <int I, int KSV, int OFF>
  SR_DEV void read(RawFrag<KMAJ>& f) const {
    if constexpr (KMAJ) {
      f.v = rd16<OFF + (I >> 1) * 64 * GK * 2>(a[I & 1][KSV]);
    } else {
      f.lo = rdtr<OFF + KSV * 16 * R * 2>(a[I][0]);
      f.hi = rdtr<OFF + KSV * 16 * R * 2 + 4 * R * 2>(a[I][0]);
    }
  }
  static constexpr int kReads = KMAJ ? NI : 2 * NI;   // LDS instructions per k-step
};

// BM x BN workgroup tile, four waves in 2 x 2, each (BM/2) x (BN/2) = MI x NJ MFMA tiles of
// 32 x 32 (v_mfma_f32_32x32x16_bf16).  NST operand stages in LDS.  Per k-tile t: k-steps
// 0..KS-2 read the next step's fragments and issue this step's MFMAs; then the wait for tile
// t+1's fill and the workgroup barrier, after which tile t's stage takes tile t+NST and tile
// t+1's first fragments are read while the last k-step's MFMAs run.  Fills are issued NST-1
// tiles ahead; fragment reads are explicit (see lds_read16), so no read waits for a fill it
// does not need.  OCC workgroups share a CU: with two, one workgroup's epilogue (GELU math,
// output stores) overlaps the other's MFMAs.
template <int BM, int BN, int NST, int OCC, bool AK, bool BK, int EPI, typename T, typename Ta>
__global__ __launch_bounds__(256, OCC) void gemm_mfma_kernel(const bf16_t* __restrict__ A, const bf16_t* __restrict__ Bm,
                                                           int M, int N, int Kd, int lda, int ldb, uint32_t a_bytes,
                                                           uint32_t b_bytes, int k_per_split, int tiles_m, int tiles_n,
                                                           EpiArgs ep) {
  constexpr int MI = BM / 64, NJ = BN / 64;
  static_assert(BM == 64 || BM == 128 || BM == 256, "tile height");
  static_assert(BN == 128 || BN == 256, "tile width");
  static_assert(NST >= 2 && NST <= 4, "stages");
  constexpr int STAGE = (BM + BN) * GK;   // bf16 elements: A tile, then B tile
  constexpr int SB = STAGE * 2;           // bytes of a stage
  constexpr int LPT = (BM + BN) / 32;     // fill instructions per thread per tile
  static_assert((NST - 1) * LPT < 64, "loads in flight exceed the vmcnt range");
  using FA = FragAddr<BM, AK, MI>;
  using FB = FragAddr<BN, BK, NJ>;
  constexpr int RPK = FA::kReads + FB::kReads;   // LDS reads per k-step
  static_assert(RPK < 16, "reads per k-step exceed the lgkmcnt range");
  __shared__ __attribute__((aligned(1024))) bf16_t smem[NST * STAGE];

  const int lane = threadIdx.x & 63, wid = wave_index();
  const int wm = wid >> 1, wn = wid & 1, h = lane >> 5;
  int tm, tn, split;
  tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn, split);
  const int m0 = tm * BM, n0 = tn * BN;
  const int kbeg = split * k_per_split;
  const int kend = min(Kd, kbeg + k_per_split);
  const int ntile = kbeg < kend ? (kend - kbeg + GK - 1) / GK : 0;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(A, a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(Bm, b_bytes);

  f32x16 acc[MI][NJ];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  TileFill<BM, AK> fla;
  TileFill<BN, BK> flb;
  fla.init(m0, lda, lane, wid);
  flb.init(n0, ldb, lane, wid);
  auto fill = [&](int t, int s) {
    bf16_t* st = smem + s * STAGE;
    const uint32_t k0 = (uint32_t)(kbeg + t * GK);
    const bool valid = t < ntile;
    fill_issue<BM / 32>(fla.off, ra, st, wid, valid ? k0 * (AK ? 2u : 2u * (uint32_t)lda) : 0x80000000u);
    fill_issue<BN / 32>(flb.off, rb, st + BM * GK, wid, valid ? k0 * (BK ? 2u : 2u * (uint32_t)ldb) : 0x80000000u);
  };
  const uint32_t sbase = lds_addr(smem);
  FA fad;
  FB fbd;
  fad.init(sbase, wm * (BM / 2), lane);
  fbd.init(sbase + BM * GK * 2, wn * (BN / 2), lane);
  RawFrag<AK> fa[2][MI];
  RawFrag<BK> fb[2][NJ];
  bf16x8 ua[MI], ub[NJ];   // settled operands of the k-step being multiplied
  // fragments of k-step KSV of stage S into buffer BUF
  auto read = [&](auto sidx, auto ksv, auto buf) {
    constexpr int S = decltype(sidx)::value, KSV = decltype(ksv)::value, BUF = decltype(buf)::value;
    static_for<MI>([&](auto i) { fad.template read<i.value, KSV, S * SB>(fa[BUF][i.value]); });
    static_for<NJ>([&](auto j) { fbd.template read<j.value, KSV, S * SB>(fb[BUF][j.value]); });
  };
  // after the wait: pin the buffer's registers and form the MFMA operands
  auto settle = [&](int buf) {
#pragma unroll
    for (int i = 0; i < MI; ++i) ua[i] = fa[buf][i].settle();
#pragma unroll
    for (int j = 0; j < NJ; ++j) ub[j] = fb[buf][j].settle();
  };
  auto mfmas = [&]() {
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ua[i], ub[j], acc[i][j], 0, 0, 0);
  };

  // EPI_DW bias gradient: row sums of A (r-major there: k-rows of BM values).  The tile row's
  // tiles_n workgroups share the work: workgroup tn sums the k-tiles t with t % tiles_n == tn.
  // Thread: chunk position cp of k-rows kg, kg + KG, ...; eight running sums.
  constexpr int CPR = BM / 8, KG = 256 / CPR;
  const bool want_db = EPI == EPI_DW && ep.db_out != nullptr;
  float dbv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const uint32_t db_addr = sbase + (uint32_t)(((threadIdx.x / CPR) * BM + (threadIdx.x % CPR) * 8) * 2);
  auto db_sum = [&](auto sidx) {
    constexpr int S = decltype(sidx)::value;
    i32x4 w[64 / KG];
    static_for<64 / KG>([&](auto j) { w[j.value] = rd16<S * SB + j.value * KG * BM * 2>(db_addr); });
    lgkm_wait<0>();
#pragma unroll
    for (int j = 0; j < 64 / KG; ++j) {
      pin(w[j]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        dbv[2 * q] += __uint_as_float((uint32_t)w[j][q] << 16);
        dbv[2 * q + 1] += __uint_as_float((uint32_t)w[j][q] & 0xFFFF0000u);
      }
    }
  };

  // prologue: tiles 0..NST-1 in flight (fills past the last k-tile read zeros), wait for tile 0
  fill(0, 0);
  fill(1, 1);
  if constexpr (NST > 2) fill(2, 2);
  if constexpr (NST > 3) fill(3, 3);
  wait_vm_lgkm0<(NST - 1) * LPT>();
  lds_barrier();
  read(IC<0>{}, IC<0>{}, IC<0>{});

  auto body = [&](int t, auto sidx) {
    constexpr int S = decltype(sidx)::value;
    if (want_db && t % tiles_n == tn) db_sum(sidx);
    static_for<KS - 1>([&](auto ksv) {
      constexpr int ks = decltype(ksv)::value;
      read(sidx, IC<ks + 1>{}, IC<(ks + 1) & 1>{});
      lgkm_wait<RPK>();   // this k-step's fragments (read one step earlier) have arrived
      settle(ks & 1);
      __builtin_amdgcn_sched_barrier(0);
      mfmas();
      __builtin_amdgcn_sched_barrier(0);
    });
    // tile t+1 resident (its fill is the oldest still in flight: every body issues exactly
    // one), every wave done reading tile t's stage
    wait_vm_lgkm0<(NST - 2) * LPT>();
    lds_barrier();
    settle((KS - 1) & 1);
    fill(t + NST, S);
    read(IC<(S + 1) % NST>{}, IC<0>{}, IC<KS & 1>{});   // unused past the last tile
    __builtin_amdgcn_sched_barrier(0);
    mfmas();
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int t = 0; t < ntile; t += NST) {
    body(t, IC<0>{});
    if (t + 1 < ntile) body(t + 1, IC<1 % NST>{});
    if constexpr (NST > 2)
      if (t + 2 < ntile) body(t + 2, IC<2 % NST>{});
    if constexpr (NST > 3)
      if (t + 3 < ntile) body(t + 3, IC<3 % NST>{});
  }
  // the last body read the next tile's first fragments, which nothing uses: keep their
  // registers allocated until the reads have landed, or the late writes could clobber
  // whatever the compiler puts there next
  lgkm_wait<0>();
  settle(KS & 1);
  wait_vm_lgkm0<0>();
  __syncthreads();   // stages free for the epilogue

  if constexpr (EPI == EPI_DW) {
    if (want_db) {
      // combine the KG partial sums of each row through LDS, in k-group order
      float* red = reinterpret_cast<float*>(smem);   // [KG][BM]
      const int cp = threadIdx.x % CPR, kg = threadIdx.x / CPR;
      const int lc = cp ^ rswz<BM>(kg);   // logical chunk this thread summed
#pragma unroll
      for (int e = 0; e < 8; ++e) red[kg * BM + lc * 8 + e] = dbv[e];
      __syncthreads();
      if ((int)threadIdx.x < BM) {
        float sum = 0.f;
        for (int g = 0; g < KG; ++g) sum += red[g * BM + threadIdx.x];
        const int row = m0 + threadIdx.x;
        const int nparts = gridDim.x / (tiles_m * tiles_n) * tiles_n;
        if (row < M) {
          if (nparts == 1) ep.db_out[row] = sum;
          else ep.dbpart[(size_t)(split * tiles_n + tn) * M + row] = sum;
        }
      }
      __syncthreads();
    }
  }

  // epilogue in MI passes of 64 rows: pass p stages i-block p of both wave rows (every wave
  // writes; register r of a 32 x 32 MFMA tile holds row 8 (r/4) + 4 h + r%4, column lane%32)
  // as fp32 in LDS, then each thread finishes NB 4-column chunks.  The epilogue's global inputs
  // (residual, GELU pre-activation, O) of every pass are loaded before the first pass and the
  // bias once, so no pass waits on a global load it issued itself.
  if constexpr (EPI == EPI_DW)
    if (gridDim.x > (unsigned)(tiles_m * tiles_n)) ep.out_f32 = ep.part + (size_t)split * ep.split_stride;
  constexpr int PR = 64;
  constexpr int EPI_LD = BN + 8;   // fp32 row stride: the two halves of a wave hit disjoint banks
  constexpr int CPRo = BN / 4;     // 4-column chunks per row
  constexpr int NB = PR * CPRo / 256;
  static_assert(256 % CPRo == 0, "a thread's chunks share their columns");
  static_assert(PR * EPI_LD * 4 <= NST * SB, "epilogue staging exceeds the stages");
  float* stg = reinterpret_cast<float*>(smem);
  // chunk q of pass p: staging row lr = c / CPRo (c = tid + 256 q), columns c4 .. c4 + 3
  auto chunk_row = [&](int p, int q) {
    const int lr = (threadIdx.x + 256 * q) / CPRo;
    return m0 + (lr >> 5) * (BM / 2) + p * 32 + (lr & 31);
  };
  const int c4 = (threadIdx.x % CPRo) * 4;
  const int n = n0 + c4;
  const f32x4 bias = n < N ? epi_bias<EPI>(ep, n) : f32x4{0.f, 0.f, 0.f, 0.f};
  EpiIn in[MI][NB];
#pragma unroll
  for (int p = 0; p < MI; ++p)
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int m = chunk_row(p, q);
      if (m < M && n < N) epi_load<EPI>(ep, m, n, in[p][q]);
    }
#pragma unroll
  for (int p = 0; p < MI; ++p) {
    if (p) __syncthreads();
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        stg[(wm * 32 + 8 * (r >> 2) + 4 * h + (r & 3)) * EPI_LD + wn * (BN / 2) + j * 32 + (lane & 31)] = acc[p][j][r];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int lr = (threadIdx.x + 256 * q) / CPRo;
      const int m = chunk_row(p, q);
      float part = 0.f;
      if (m < M && n < N)
        part = epi_store<EPI>(ep, m, n, *reinterpret_cast<const f32x4*>(stg + lr * EPI_LD + c4), in[p][q], bias);
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

// Sum of split-K partial planes, in split order: out[i] = sum_z part[z * n + i] (float4 lanes),
// and of the bias-gradient partial rows: dbout[c] = sum_z dbpart[z * nb + c].
__global__ __launch_bounds__(256) void reduce_splits_kernel(const float* __restrict__ part, int splits, size_t n4,
                                                            float* __restrict__ out, const float* __restrict__ dbpart,
                                                            int dbparts, int nb, float* __restrict__ dbout) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n4) {
    const f32x4* p = reinterpret_cast<const f32x4*>(part);
    f32x4 s = p[i];
    for (int z = 1; z < splits; ++z) s += p[(size_t)z * n4 + i];
    reinterpret_cast<f32x4*>(out)[i] = s;
  } else if (dbout && i - n4 < (size_t)nb) {
    const size_t c = i - n4;
    float s = dbpart[c];
    for (int z = 1; z < dbparts; ++z) s += dbpart[(size_t)z * nb + c];
    dbout[c] = s;
  }
}

// Several reductions in one launch (the reductions of one block's backward): job j takes blocks
// [first[j], first[j + 1]).  A split-K / bias job does exactly what reduce_splits_kernel does for
// it (one f32x4 or one bias column per thread); a column-sum job covers 64 columns per block
// with 16 row phases, exactly as reduce_cols_kernel (summed over all rows, no accumulation).
struct ReduceJobs {
  ReduceJob job[kMaxReduceJobs];
  int first[kMaxReduceJobs + 1];
};
constexpr int kReduceJobThreads = 1024;
__global__ __launch_bounds__(kReduceJobThreads) void reduce_jobs_kernel(ReduceJobs rj) {
  __shared__ float red[16][65];
  int j = 0;
  while (j + 1 < kMaxReduceJobs && (int)blockIdx.x >= rj.first[j + 1]) ++j;
  const ReduceJob& b = rj.job[j];
  const int blk = (int)blockIdx.x - rj.first[j];
  if (b.rows > 0) {   // uniform over the block (one job per block)
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const int c = blk * 64 + tx;
    float acc = 0.f;
    if (c < b.width) {
      int rr = ty;
      for (; rr + 7 * 16 < b.rows; rr += 8 * 16) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = b.part[(size_t)(rr + i * 16) * b.width + c];
#pragma unroll
        for (int i = 0; i < 8; ++i) acc += v[i];
      }
      for (; rr < b.rows; rr += 16) acc += b.part[(size_t)rr * b.width + c];
    }
    red[ty][tx] = acc;
    __syncthreads();
    for (int s = 8; s >= 1; s >>= 1) {
      if (ty < s) red[ty][tx] += red[ty + s][tx];
      __syncthreads();
    }
    if (ty == 0 && c < b.width) {
      float* o = c < b.half ? (b.out ? b.out + c : nullptr) : (b.dbout ? b.dbout + (c - b.half) : nullptr);
      if (o) *o = red[0][tx];
    }
    return;
  }
  const size_t n4 = b.splits > 1 ? b.n / 4 : 0;
  const size_t i = (size_t)blk * kReduceJobThreads + threadIdx.x;
  if (i < n4) {
    const f32x4* p = reinterpret_cast<const f32x4*>(b.part);
    f32x4 s = p[i];
    for (int z = 1; z < b.splits; ++z) s += p[(size_t)z * n4 + i];
    reinterpret_cast<f32x4*>(b.out)[i] = s;
  } else if (b.dbout && i - n4 < (size_t)b.nb) {
    const size_t c = i - n4;
    float s = b.dbpart[c];
    for (int z = 1; z < b.dbparts; ++z) s += b.dbpart[(size_t)z * b.nb + c];
    b.dbout[c] = s;
  }
}

hipError_t launch_reduce_jobs(const ReduceJob* jobs, int njobs, hipStream_t st) {
  ReduceJobs rj{};
  int blocks = 0, k = 0;
  for (int j = 0; j < njobs; ++j) {
    const ReduceJob& b = jobs[j];
    int nblk;
    if (b.rows > 0) {
      nblk = (b.out || b.dbout) && b.width > 0 ? (b.width + 63) / 64 : 0;
    } else {
      const size_t total = (b.splits > 1 ? b.n / 4 : 0) + (b.dbout ? b.nb : 0);
      nblk = (int)((total + kReduceJobThreads - 1) / kReduceJobThreads);
    }
    if (nblk == 0) continue;
    if (k == kMaxReduceJobs) return hipErrorInvalidValue;   // more jobs than one launch holds
    rj.job[k] = b;
    rj.first[k] = blocks;
    blocks += nblk;
    ++k;
  }
  if (blocks == 0) return hipSuccess;
  for (int j = k; j <= kMaxReduceJobs; ++j) rj.first[j] = blocks;
  SR_LAUNCH(reduce_jobs_kernel, dim3((unsigned)blocks), dim3(kReduceJobThreads), 0, st, rj);
  return hipGetLastError();
}

static hipError_t launch_reduce(const float* part, int splits, size_t n, float* out, const float* dbpart, int dbparts,
                                int nb, float* dbout, hipStream_t st) {
  const size_t n4 = splits > 1 ? n / 4 : 0;
  const size_t total = n4 + (dbout ? nb : 0);
  if (total == 0) return hipSuccess;
  SR_LAUNCH(reduce_splits_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, part, splits, n4,
                     out, dbpart, dbparts, nb, dbout);
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

// Tile shapes of the MFMA kernel, with the stage count that fits the 160 KB of LDS.
enum TileShape { T256x256 = 0, T256x128 = 1, T128x256 = 2, T128x128 = 3, T64x128 = 4, T128x128x2 = 5 };

template <int BM, int BN, int NST, int OCC, int EPI, typename T, typename Ta>
static hipError_t run_mfma_tile(const GemmDesc& g, const EpiArgs& ep, int splits, int kps, hipStream_t st) {
  const int tiles_m = (g.M + BM - 1) / BM, tiles_n = (g.N + BN - 1) / BN;
  const dim3 grid((unsigned)(tiles_m * tiles_n * splits));
#define SR_GEMM_L(AK, BK)                                                                                        \
  SR_LAUNCH((gemm_mfma_kernel<BM, BN, NST, OCC, AK, BK, EPI, T, Ta>), grid, dim3(256), 0, st,            \
                     (const bf16_t*)g.A, (const bf16_t*)g.B, g.M, g.N, g.K, (int)g.lda, (int)g.ldb,               \
                     (uint32_t)g.a_bytes, (uint32_t)g.b_bytes, kps, tiles_m, tiles_n, ep)
  if (g.a_kmajor && g.b_kmajor) SR_GEMM_L(true, true);
  else if (g.a_kmajor && !g.b_kmajor) SR_GEMM_L(true, false);
  else if (!g.a_kmajor && !g.b_kmajor) SR_GEMM_L(false, false);
  else SR_GEMM_L(false, true);
#undef SR_GEMM_L
  return hipGetLastError();
}

template <int EPI, typename T, typename Ta>
static hipError_t run_shape(int shape, const GemmDesc& g, const EpiArgs& ep, int splits, int kps, hipStream_t st) {
  switch (shape) {
    case T256x128: return run_mfma_tile<256, 128, 3, 1, EPI, T, Ta>(g, ep, splits, kps, st);
    case T128x256: return run_mfma_tile<128, 256, 3, 1, EPI, T, Ta>(g, ep, splits, kps, st);
    case T128x128: return run_mfma_tile<128, 128, 4, 1, EPI, T, Ta>(g, ep, splits, kps, st);
    case T128x128x2: return run_mfma_tile<128, 128, 2, 2, EPI, T, Ta>(g, ep, splits, kps, st);
    default: return run_mfma_tile<64, 128, 4, 1, EPI, T, Ta>(g, ep, splits, kps, st);
  }
}

static int shape_bm(int s) { return s == T256x256 || s == T256x128 ? 256 : s == T64x128 ? 64 : 128; }
static int shape_occ(int s) { return s == T128x128x2 ? 2 : 1; }
static int shape_bn(int s) { return s == T256x256 || s == T128x256 ? 256 : 128; }

// Tile shape by the number of 128 x 128 output tiles (measured on the block's GEMMs at 4050
// tokens on MI355X): many tiles -> two 128 x 128 workgroups per CU (one's epilogue overlaps the
// other's MFMAs); about one per CU -> one workgroup with a four-stage pipeline; fewer -> 64 x 128
// tiles so that the grid still covers the CUs.  The 256 x 128 shapes measured slower throughout
// and stay available to the benchmarks only.
static int pick_shape(int M, int N, int splits) {
  const long tiles = (long)((M + 127) / 128) * ((N + 127) / 128) * splits;
  if (tiles >= 384) return T128x128x2;
  if (tiles >= 192) return T128x128;
  return T64x128;
}

#ifdef SR_GEMM_FORCE_SHAPE
int g_force_shape = -1;   // standalone benchmarks: >= 0 overrides the choice
#endif

template <int EPI, typename T, typename Ta>
static hipError_t run_mfma(const GemmDesc& g, const EpiArgs& ep, hipStream_t st) {
  const int splits = g.splits > 1 ? g.splits : 1;
  const int kps = splits > 1 ? g.k_per_split : g.K;
  int shape = pick_shape(g.M, g.N, splits);
#ifdef SR_GEMM_FORCE_SHAPE
  if (g_force_shape >= 0) shape = g_force_shape;
#endif
  return run_shape<EPI, T, Ta>(shape, g, ep, splits, kps, st);
}

// Weight gradient (EPI_DW; reduction over tokens, both operands r-major): shape and split-K
// factor.  Few output tiles are split over tokens so that the grid covers the GPU; each split
// writes a partial plane that one reduction adds in split order.
struct DwPlan {
  int shape, splits, kps, tiles_n;
};
static DwPlan dw_plan(int M, int N, int K) {
  DwPlan p;
  p.shape = pick_shape(M, N, 1);
#ifdef SR_GEMM_FORCE_SHAPE
  if (g_force_shape >= 0) p.shape = g_force_shape;
#endif
  const int bm = shape_bm(p.shape), bn = shape_bn(p.shape);
  const long tiles = (long)((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  int sp = (int)(256 * shape_occ(p.shape) / tiles);   // one round of workgroups at most
  sp = std::min(sp, std::max(1, K / 512));
  sp = std::max(1, std::min(sp, 8));
  p.kps = ((K + sp - 1) / sp + GK - 1) / GK * GK;
  p.splits = (K + p.kps - 1) / p.kps;
  if (p.splits <= 1) { p.splits = 1; p.kps = K; }
  p.tiles_n = (N + bn - 1) / bn;
  return p;
}

template <int EPI, typename T, typename Ta, typename TA, typename TB>
static hipError_t run_simple(const GemmDesc& g, const EpiArgs& ep, hipStream_t st) {
  dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, 1);
  const long long a_sm = g.a_kmajor ? g.lda : 1, a_sk = g.a_kmajor ? 1 : g.lda;
  const long long b_sn = g.b_kmajor ? g.ldb : 1, b_sk = g.b_kmajor ? 1 : g.ldb;
  SR_LAUNCH((gemm_simple_kernel<TA, TB, EPI, T, Ta>), grid, dim3(256), 0, st, (const TA*)g.A,
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
    case EPI_DW: return g.use_mfma ? hipErrorInvalidValue : dispatch<EPI_DW>(g, ep, st);   // launch_weight_grad
    case EPI_DO: return g.use_mfma ? run_mfma<EPI_DO, bf16_t, bf16_t>(g, ep, st) : hipErrorInvalidValue;
  }
  return hipErrorInvalidValue;
}

// gz = Ta(GELU(z)) from the stored FC1 pre-activation: the FC1 epilogue's values, recomputed for
// the FC2 weight gradient instead of being kept from the forward.  Eight elements per thread.
template <typename Ta>
__global__ __launch_bounds__(256) void gelu_kernel(const Ta* __restrict__ z, Ta* __restrict__ gz, size_t n8) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (size_t)gridDim.x * 256) {
    if constexpr (sizeof(Ta) == 2) {
      const i32x4 w = reinterpret_cast<const i32x4*>(z)[i];
      i32x4 out;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        i32x2 zb;
        zb[0] = w[2 * h];
        zb[1] = w[2 * h + 1];
        const f32x4 zf = unpack4(zb);
        f32x4 g;
#pragma unroll
        for (int q = 0; q < 4; ++q) g[q] = gelu_f<gelu_deg<Ta>()>(zf[q]);
        const i32x2 gb = pack4(g);
        out[2 * h] = gb[0];
        out[2 * h + 1] = gb[1];
      }
      reinterpret_cast<i32x4*>(gz)[i] = out;
    } else {
#pragma unroll
      for (int q = 0; q < 8; ++q) gz[8 * i + q] = gelu_f<gelu_deg<Ta>()>(z[8 * i + q]);
    }
  }
}

hipError_t launch_gelu(int dtype, const void* z, void* gz, size_t n, hipStream_t st) {
  const size_t n8 = n / 8;   // n is a multiple of 64 (F % 64 == 0)
  const dim3 g((unsigned)std::min<size_t>((n8 + 255) / 256, 4096));
  if (dtype == kBF16)
    SR_LAUNCH(gelu_kernel<bf16_t>, g, dim3(256), 0, st, (const bf16_t*)z, (bf16_t*)gz, n8);
  else
    SR_LAUNCH(gelu_kernel<float>, g, dim3(256), 0, st, (const float*)z, (float*)gz, n8);
  return hipGetLastError();
}

void weight_grad_scratch(int M, int N, int K, size_t* part_floats, size_t* dbpart_floats) {
  const DwPlan p = dw_plan(M, N, K);
  *part_floats = p.splits > 1 ? (size_t)p.splits * M * N : 0;
  *dbpart_floats = (size_t)p.splits * p.tiles_n * M;
}

hipError_t launch_weight_grad(const GemmDesc& g, float* dw, float* db, float* part, float* dbpart, hipStream_t st,
                              ReduceJob* defer) {
  if (defer) *defer = ReduceJob{};
  EpiArgs ep;
  ep.ldo = g.N;
  if (!g.use_mfma) {
    ep.out_f32 = dw;
    ep.db_out = db;
    return dispatch<EPI_DW>(g, ep, st);
  }
  const DwPlan p = dw_plan(g.M, g.N, g.K);
  const int nparts = p.splits * p.tiles_n;
  ep.out_f32 = dw;
  ep.part = part;
  ep.split_stride = (long long)g.M * g.N;
  ep.db_out = db;
  ep.dbpart = dbpart;
  hipError_t e = run_shape<EPI_DW, bf16_t, bf16_t>(p.shape, g, ep, p.splits, p.kps, st);
  if (e != hipSuccess) return e;
  if (p.splits > 1 || (db && nparts > 1)) {
    if (defer) {
      *defer = ReduceJob{part, p.splits, (size_t)g.M * g.N, dw, dbpart, nparts, g.M, nparts > 1 ? db : nullptr};
      return hipSuccess;
    }
    return launch_reduce(part, p.splits, (size_t)g.M * g.N, dw, dbpart, nparts, g.M, nparts > 1 ? db : nullptr, st);
  }
  return hipSuccess;
}

}  // namespace sr
