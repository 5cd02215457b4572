// Multi-head self-attention of the block (Sec. 3.3): per sample and head,
// O = softmax(q k^T / sqrt(hd)) v over all S tokens (no mask), and its backward.
//
// Layouts: qkv is token-major [B*S, 3D] (q at column h*hd, k at D + h*hd, v at
// 2D + h*hd); O and dO are [B*S, D]; dqkv mirrors qkv.  lse[b,h,s] is the base-2
// log-sum-exp of the scaled scores, so P = exp2(s * log2(e)/sqrt(hd) - lse).
//
// MFMA kernels (head dim 64 or 128, bf16, v_mfma_f32_32x32x16_bf16).  A workgroup of NW
// waves owns 32 NW rows (32 per wave) of the resident dimension and streams the other one in
// 64-row tiles of one head:
//  * forward: a wave owns 32 queries and forms S^T = K Q^T per 32-key unit, so each
//    lane holds one query's scores and the online-softmax state is per lane; the row
//    max needs one exchange between the wave's two halves (v_permlane32_swap).
//    O^T += V^T P^T reuses the score registers as the MFMA B operand (the k order inside
//    an MFMA is free as long as A and B agree).  The S x S matrix is never stored.
//  * backward dK/dV: a wave owns 32 keys; per 32-query unit S = Q K^T and dP = dO V^T
//    (key per lane), P = exp2(S c - lse), dS = P (dP - delta), dV^T += dO^T P and
//    dK^T += Q^T dS.
//  * backward dQ: a wave owns 32 queries; per 32-key unit S^T, dP^T and dQ^T += K^T dS^T.
// Two backward passes (instead of atomics) keep the result deterministic.
//  * column sums of P (the attention each key receives, for the attention-score selector of
//    Sec. 4.4): the dK/dV kernel's score half.
//
// Tiles go from global memory straight into LDS (buffer_load ... lds), three stages deep
// (tile t+2 is in flight while tile t is consumed), row-major with an XOR swizzle of the
// 16-byte chunks; one workgroup barrier per tile.  Operands needed transposed (V^T, Q^T,
// dO^T, K^T) are read with ds_read_b64_tr_b16, which hands each lane four consecutive rows
// of one column, so no transposed copy is ever written.
//
// Generic kernels (fp32 storage, or bf16 at head dim 32): one thread per row, online softmax
// over keys, fp32 throughout.
#include <type_traits>

#include "common.h"
#include "profile.h"
#include "sr_internal.h"

namespace sr {

constexpr int KT = 64;       // tile of the streamed dimension
constexpr int NSTG = 3;      // LDS stages
// Waves per workgroup of the MFMA kernels at head dim 64: eight (256 rows) share each streamed
// tile in LDS, at one workgroup per CU and two waves per SIMD; against four, measured 2-4 %
// faster per kernel at 4050 tokens (forward 94 -> 90, dK/dV 159 -> 155, dQ 112 -> 108 us).  At
// head dim 128 the accumulators of a 32-row unit take twice the registers, so four waves (128
// rows) per workgroup, one per SIMD with the whole register file: the register-explicit kernels
// attn_fwd_h128, attn_bwd_dkv_h128 and attn_bwd_dq_h128 (the templates below are instantiated at
// head dim 64).
template <int HD>
constexpr int attn_waves() { return HD == 64 ? 8 : 4; }

// Geometry of a 64-row tile of one head (head dim HD, bf16).
template <int HD>
struct Geo {
  static_assert(HD == 64 || HD == 128, "MFMA attention head dims");
  static constexpr int AP = HD + 8;     // padded row (bf16) of the output staging tile
  static constexpr int TE = KT * HD;    // bf16 elements of one 64-row tile
  static constexpr int TB = TE * 2;     // bytes of one tile
  static constexpr int SGB = 2 * TB;    // bytes of one stage (two tiles)
  static constexpr int KS = HD / 16;    // MFMA k-steps over the head dimension
  static constexpr int DB = HD / 32;    // 32-column blocks of the head dimension
  static constexpr int CPR = HD / 8;    // 16-byte chunks per row
  static constexpr int BLK = HD / 8;    // 1 KB blocks of a tile
};


SR_DEV bf16x8 zero8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
  return z;
}

SR_DEV bf16x8 ld8(const bf16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }
// sign flip of eight bf16 values (exact)
SR_DEV bf16x8 neg8(bf16x8 v) {
  i32x4 w = __builtin_bit_cast(i32x4, v);
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] ^= (int)0x80008000u;
  return __builtin_bit_cast(bf16x8, w);
}

SR_DEV f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) { return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0); }

// 2^x on the hardware unit directly: the softmax arguments are <= 0 (or -inf), where the
// unscaled instruction is accurate to ~1 ulp and flushes tiny results to zero.
SR_DEV float ex2(float x) { return __builtin_amdgcn_exp2f(x); }

SR_DEV void zero16(f32x16& a) {
#pragma unroll
  for (int r = 0; r < 16; ++r) a[r] = 0.f;
}

// LDS tile: 64 rows of HD bf16 (HD / 8 16-byte chunks each); chunk c of row r sits at chunk
// position c ^ swz(r).  The LDS serves 256 bytes (64 banks) per pass.
//  * HD = 64 (128-byte rows): among any 16 consecutive rows the even ones use eight different
//    positions and so do the odd ones (conflict-free 16-byte fragment reads); rows r and r+2 of
//    each group of four differ in bit 2 of the position, so the four rows x 64 bytes that half
//    a wave's transposed read touches fall in different banks (measured conflict-free for both
//    read kinds, where plain XOR swizzles within 64-byte groups cost one extra pass per
//    transposed read).
//  * HD = 128 (256-byte rows, each one whole pass of the banks): 16 consecutive rows take 16
//    different positions (16-byte fragment reads of 16 lanes cover every bank once), and bits
//    2-3 of the position follow the row mod 4, so the four rows x 64 bytes of a half-wave's
//    transposed read land in four different 64-byte quarters.
// Rows 16 apart share a swizzle, so fragment addresses of different 16-row groups differ by
// constants (instruction offsets rather than address registers).
template <int HD>
SR_DEV int swz(int row) {
  if constexpr (HD == 64) return (((row >> 1) & 1) << 2) | ((row >> 2) & 3);
  else return ((row & 3) << 2) | ((row >> 2) & 3);
}
template <int HD>
SR_DEV int toff(int row, int chunk) { return row * HD + ((chunk ^ swz<HD>(row)) << 3); }

// Rows r0..r0+63 of one head (columns base.. of a row-major tensor with row length ld)
// into the LDS tile dst: HD / 8 blocks of 1 KB (64 / (HD / 8) rows each); lane l lands at
// byte 16 l of its block, so it fetches the chunk that the swizzle places there.  Rows past
// the sample's S tokens are read without a guard: they belong to the next sample (finite
// values the callers mask) or lie past the tensor, where the buffer load returns zero.
// NW waves share the blocks.
template <int HD, int NW>
SR_DEV void tile_load(__amdgpu_buffer_rsrc_t rs, uint32_t base, uint32_t ld, int r0, bf16_t* dst, bool valid = true) {
  using G = Geo<HD>;
  static_assert(G::BLK % NW == 0, "tile blocks per wave");
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  constexpr int PER = G::BLK / NW, RPB = 64 / G::CPR;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int blk = wid * PER + i;
    const int row = blk * RPB + lane / G::CPR;
    const int c = (lane % G::CPR) ^ swz<HD>(row);
    uint32_t off = base + ((uint32_t)(r0 + row) * ld + (uint32_t)c * 8u) * 2u;
    // a load past the last tile keeps the number of loads in flight uniform: it reads beyond
    // every tensor's extent (2 GiB at most), which returns zeros without a memory access
    if (!valid) off = 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_ptr_t*)(dst + blk * 512), 16, off, 0, 0, 0);
  }
}

// Fragment of the 32 rows r0.. (MFMA row index = lane % 32), k-step ks of the HD columns.
template <int HD>
SR_DEV bf16x8 row_frag(const bf16_t* tile, int r0, int ks) {
  const int lane = threadIdx.x & 63;
  return ld8(tile + toff<HD>(r0 + (lane & 31), 2 * ks + (lane >> 5)));
}

// Transposed fragment: MFMA row index = tile column c0 + lane % 32, k = tile rows, in the
// order of a score fragment: elements 0..3 are rows k0 + 4h .. k0 + 4h + 3 and elements
// 4..7 rows k0 + 8 + 4h .. (h = lane / 32).  ds_read_b64_tr_b16 gives lane i of each
// 16-lane group column i of the four rows addressed by the group (lane s: row s / 4,
// columns 4 (s % 4) .. + 3).
template <int HD>
SR_DEV bf16x8 tr_frag(const bf16_t* tile, int k0, int c0) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, s = lane & 15;
  const int col = c0 + 16 * (g & 1) + 4 * (s & 3);
  const int r1 = k0 + 4 * (g >> 1) + (s >> 2), r2 = r1 + 8;
  const v4s lo = ds_tr(tile + r1 * HD + (((col >> 3) ^ swz<HD>(r1)) << 3) + (col & 7));
  const v4s hi = ds_tr(tile + r2 * HD + (((col >> 3) ^ swz<HD>(r2)) << 3) + (col & 7));
  i32x4 w;
  w[0] = __builtin_bit_cast(i32x2, lo)[0];
  w[1] = __builtin_bit_cast(i32x2, lo)[1];
  w[2] = __builtin_bit_cast(i32x2, hi)[0];
  w[3] = __builtin_bit_cast(i32x2, hi)[1];
  return __builtin_bit_cast(bf16x8, w);
}

// Explicit fragment reads (see lds_read16) from one LDS array of NSTG stages, each holding two
// 64 x HD tiles (tile p of stage s at byte offset (2 s + p) TB): per-lane base addresses are
// fixed, and the stage, tile, row-group and k-step offsets are instruction immediates.  The
// compiler then neither waits for fills in flight into other stages nor keeps per-stage
// address registers; the kernels wait (lgkm_wait) before using what they read.

// Row fragment: MFMA row index = tile row R0 + lane % 32 (R0 a multiple of 16, which keeps
// the swizzle), k-step KSV of the HD columns.
template <int HD>
struct RowAddr {
  uint32_t a[HD / 16];
  SR_DEV void init(uint32_t base, int lane) {
    const int l32 = lane & 31, h = lane >> 5;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks)
      a[ks] = base + (uint32_t)(l32 * HD + (((2 * ks + h) ^ swz<HD>(l32)) << 3)) * 2u;
  }
  template <int OFF, int R0, int KSV>
  SR_DEV void read(RawFrag<true>& f) const {
    f.v = rd16<OFF + R0 * HD * 2>(a[KSV]);
  }
};

// Transposed fragment (as tr_frag): MFMA row index = tile column 32 DBV + lane % 32, k = tile
// rows K0 + 4 h .. + 3 (first read) and K0 + 8 + 4 h .. + 3 (second read), K0 a multiple of 16.
template <int HD>
struct TrAddr {
  uint32_t a[HD / 32][2];
  SR_DEV void init(uint32_t base, int lane) {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) {
      const int col = 32 * db + 16 * (g & 1) + 4 * (s & 3);
      const int r1 = 4 * (g >> 1) + (s >> 2), r2 = r1 + 8;
      a[db][0] = base + (uint32_t)(r1 * HD + (((col >> 3) ^ swz<HD>(r1)) << 3) + (col & 7)) * 2u;
      a[db][1] = base + (uint32_t)(r2 * HD + (((col >> 3) ^ swz<HD>(r2)) << 3) + (col & 7)) * 2u;
    }
  }
  template <int OFF, int K0, int DBV>
  SR_DEV void read(RawFrag<false>& f) const {
    f.lo = rdtr<OFF + K0 * HD * 2>(a[DBV][0]);
    f.hi = rdtr<OFF + K0 * HD * 2>(a[DBV][1]);
  }
};

// Row index (within a 32-row unit) of score register r of this lane.
SR_DEV int srow(int r, int h32) { return 8 * (r >> 2) + 4 * h32 + (r & 3); }

// Write a wave's 32 x HD result (held transposed: acc[db][r] = X[d][row]) to LDS
// stage[row_local][d], scaled.
template <int HD>
SR_DEV void stage_t(bf16_t* stage, const f32x16 acc[HD / 32], float mul, int wid, int lane) {
  const int l32 = lane & 31, h32 = lane >> 5;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      stage[(wid * 32 + l32) * Geo<HD>::AP + db * 32 + srow(r, h32)] = f2bf(acc[db][r] * mul);
}

// Copy the (32 NW) x HD staged tile to rows r0.. of dst (column block of one head); NW waves.
template <int HD, int NW>
SR_DEV void unstage(const bf16_t* stage, bf16_t* dst, size_t ld, int r0, int S) {
  constexpr int CPR = Geo<HD>::CPR;
#pragma unroll
  for (int i = 0; i < CPR / 2; ++i) {
    const int c = threadIdx.x + 64 * NW * i;
    const int row = c / CPR, kc = c % CPR;
    if (r0 + row < S)
      *reinterpret_cast<i32x4*>(dst + (size_t)(r0 + row) * ld + kc * 8) =
          *reinterpret_cast<const i32x4*>(stage + row * Geo<HD>::AP + kc * 8);
  }
}

// Workgroups go to the eight XCDs in dispatch order round-robin (linear id mod 8), and each XCD
// has its own L2.  The MFMA kernels remap their ids so that the workgroups of one (sample, head)
// pair -- which all stream the same tiles -- run on one XCD: dispatch slot s of XCD x takes the
// (x N / 8 + s)-th (block, head, sample) triple in block-fastest order.  Identity when the
// grid's size N is not a multiple of 8.
struct TileId {
  int blk, h, b;
};
SR_DEV TileId xcd_tile_id() {
  const int nb = gridDim.x, nh = gridDim.y, n = nb * nh * gridDim.z;
  int l = blockIdx.x + nb * (blockIdx.y + nh * blockIdx.z);
  if ((n & 7) == 0) l = (l & 7) * (n >> 3) + (l >> 3);
  return {l % nb, (l / nb) % nh, l / (nb * nh)};
}

// ------------------------------------------------------------------------------ forward

// NW waves (32 queries each) per workgroup share the K / V tiles.
// Queries: Sq rows of q (row stride ldq); keys: Skv rows of kv (row stride ldkv), values D
// columns after the keys; kv_elems: elements addressable from kv (the buffer's extent).
template <int HD, int NW>
__global__ __launch_bounds__(64 * NW, HD == 64 ? 8 / NW : 1) void attn_fwd_mfma(const bf16_t* __restrict__ q, int ldq,
                                                     const bf16_t* __restrict__ kv, int ldkv, uint32_t kv_elems,
                                                     bf16_t* __restrict__ O, float* __restrict__ lse, int Sq, int Skv,
                                                     int H, int D, float sl2) {
  using G = Geo<HD>;
  constexpr int TE = G::TE, TB = G::TB, SGB = G::SGB, KS = G::KS, DB = G::DB;
  __shared__ __attribute__((aligned(16))) bf16_t smem[NSTG * 2 * TE];   // stage: K tile, V tile
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const bf16_t* qp = q + (size_t)b * Sq * ldq + hh * HD;
  const int myq = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (Skv + KT - 1) / KT;
  const bool ragged = Skv % KT != 0;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(kv, kv_elems * 2u);
  const uint32_t kbase = (uint32_t)(((size_t)b * Skv * ldkv + hh * HD) * 2);
  const uint32_t vbase = kbase + (uint32_t)D * 2u;
  RowAddr<HD> ra;
  TrAddr<HD> ta;
  ra.init(lds_addr(smem), lane);
  ta.init(lds_addr(smem), lane);

  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = myq < Sq ? ld8(qp + (size_t)myq * ldq + ks * 16 + 8 * h32) : zero8();

  constexpr int kLoads = 2 * (G::BLK / NW);   // buffer loads per thread per tile (two tiles)
  auto load = [&](int t, int s) {
    tile_load<HD, NW>(rq, kbase, (uint32_t)ldkv, t * KT, smem + s * 2 * TE, t < nt);
    tile_load<HD, NW>(rq, vbase, (uint32_t)ldkv, t * KT, smem + s * 2 * TE + TE, t < nt);
  };
  auto mask = [&](f32x16& sc, int k0) {   // keys past Skv do not exist
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (k0 + srow(r, h32) >= Skv) sc[r] = -INFINITY;
  };

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) zero16(o[db]);
  // softmax denominators on the matrix cores: a 32-row A operand whose row 0 is all ones turns
  // the P^T MFMA into the column sums of P^T, so lsum[0] of lane l32 (first half) is the sum of
  // the bf16 probabilities of query l32 (the values the PV product uses); every other element
  // stays zero
  f32x16 lsum;
  zero16(lsum);
  bf16x8 ones;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones[i] = (__bf16)(l32 == 0 ? 1.0f : 0.0f);
  float m_run = -INFINITY;   // running max of the raw scores
  // K row fragments of key unit U of stage SG
  auto read_k = [&](auto sg, auto uu, RawFrag<true> (&kr)[KS]) {
    constexpr int SG = decltype(sg)::value, U = decltype(uu)::value;
    static_for<KS>([&](auto ks) { ra.template read<SG * SGB, U * 32, decltype(ks)::value>(kr[ks.value]); });
  };
  // S^T = K Q^T of a unit: register r holds key srow(r), query l32
  auto scores = [&](RawFrag<true> (&kr)[KS], f32x16& sc) {
    zero16(sc);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) sc = mfma(kr[ks].settle(), qf[ks], sc);
  };
  // V^T fragments of unit U (read before the softmax arithmetic, so that their latency hides
  // behind it)
  auto read_vt = [&](auto sg, auto uu, RawFrag<false> (&vt)[DB][2]) {
    constexpr int SG = decltype(sg)::value, U = decltype(uu)::value;
    static_for<DB>([&](auto db) {
      static_for<2>([&](auto kk) {
        ta.template read<SG * SGB + TB, U * 32 + decltype(kk)::value * 16, decltype(db)::value>(vt[db.value][kk.value]);
      });
    });
  };
  // online softmax over the tile's 64 keys (one reference update for both units), then
  // O^T += V^T P^T per unit
  auto consume = [&](auto sg, const f32x16& sc0, const f32x16& sc1) {
    RawFrag<false> vt0[DB][2], vt1[DB][2];
    read_vt(sg, IC<0>{}, vt0);
    read_vt(sg, IC<1>{}, vt1);
    float mx = fmaxf(sc0[0], sc1[0]);
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, fmaxf(sc0[r], sc1[r]));
    mx = half_pair_max(mx);
    // lazy rescaling: the reference max m_run moves (and O, l are rescaled) only when a
    // row's max has grown by more than 8 in exp2 units; otherwise p = 2^((s - m_run) c) <= 256,
    // and since O and l share the reference the result is the same
    const float grow = (fmaxf(m_run, mx) - m_run) * sl2;   // +inf on the first tile
    if (__ballot(grow > 8.0f)) {
      const float m_ref = grow > 8.0f ? mx : m_run;
      const float alpha = ex2((m_run - m_ref) * sl2);
      lsum[0] *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      m_run = m_ref;
    }
    const float nm = -m_run * sl2;
    bf16x8 pb0[2], pb1[2];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      pb0[r >> 3][r & 7] = (__bf16)ex2(fmaf(sc0[r], sl2, nm));
      pb1[r >> 3][r & 7] = (__bf16)ex2(fmaf(sc1[r], sl2, nm));
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      lsum = mfma(ones, pb0[kk], lsum);
      lsum = mfma(ones, pb1[kk], lsum);
    }
    lgkm_wait<0>();
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        o[db] = mfma(vt0[db][kk].settle(), pb0[kk], o[db]);
        o[db] = mfma(vt1[db][kk].settle(), pb1[kk], o[db]);
      }
  };

  load(0, 0);
  load(1, 1);   // past the last tile: zeros (a uniform count of loads in flight)
  wait_vm_lgkm0<kLoads>();
  lds_barrier();
  auto tile = [&](int t, auto stg) {
    constexpr int s0 = decltype(stg)::value;
    const bool rag = ragged && t + 1 == nt;
    // tile t+2 into the stage of tile t-1, which every wave has left (the barrier that ended
    // tile t-1); it then flies during tiles t and t+1
    load(t + 2, (s0 + 2) % NSTG);
    // both units' score MFMAs first: unit 1's run while unit 0's softmax arithmetic does
    RawFrag<true> k0r[KS], k1r[KS];
    f32x16 sc0, sc1;
    read_k(stg, IC<0>{}, k0r);
    read_k(stg, IC<1>{}, k1r);
    lgkm_wait<0>();
    scores(k0r, sc0);
    scores(k1r, sc1);
    if (rag) {
      if (Skv - t * KT < 32) mask(sc0, t * KT);
      if (Skv - t * KT < 64) mask(sc1, t * KT + 32);
    }
    consume(stg, sc0, sc1);
    wait_vm_lgkm0<kLoads>();   // tile t+1 resident: only tile t+2's loads may still fly
    lds_barrier();             // ... for every wave, and every wave is done with tile t's stage
  };
  int t = 0;
  for (; t + NSTG <= nt; t += NSTG) {
    tile(t, IC<0>{});
    tile(t + 1, IC<1>{});
    tile(t + 2, IC<2>{});
  }
  if (t < nt) tile(t, IC<0>{});
  if (t + 1 < nt) tile(t + 1, IC<1>{});

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();   // every wave is done with the stages before they hold the output
  const float l_tot = half_pair_sum(lsum[0]);   // the second half's element is zero
  if (h32 == 0 && myq < Sq) lse[((size_t)b * H + hh) * Sq + myq] = m_run * sl2 + log2f(l_tot);
  stage_t<HD>(smem, o, 1.0f / l_tot, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, O + (size_t)b * Sq * D + hh * HD, D, id.blk * (32 * NW), Sq);
}

// ------------------------------------------------------------------------------ backward dK, dV

// NW waves (32 keys each) per workgroup share the Q / dO tiles.
template <int HD, int NW>
// Keys: Skv rows of kv (stride ldkv, values D columns on); queries: Sq rows of q (stride ldq,
// q_elems addressable elements); dK to dk_out (stride ldo), dV D columns after it.
__global__ __launch_bounds__(64 * NW, HD == 64 ? 8 / NW : 1) void attn_bwd_dkv_mfma(const bf16_t* __restrict__ q, int ldq,
                                                         uint32_t q_elems, const bf16_t* __restrict__ kv, int ldkv,
                                                         const bf16_t* __restrict__ dO,
                                                         const float* __restrict__ lse, const float* __restrict__ delta,
                                                         bf16_t* __restrict__ dk_out, int ldo, int Sq, int Skv, int H,
                                                         int D, float sl2, float scale) {
  using G = Geo<HD>;
  constexpr int TE = G::TE, KS = G::KS, DB = G::DB;
  __shared__ __attribute__((aligned(16))) bf16_t smem[NSTG * 2 * TE];   // stage: Q tile, dO tile
  __shared__ __attribute__((aligned(16))) float fsm[NSTG * 2 * KT];     // stage: lse, delta of the tile's rows
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const bf16_t* kp = kv + (size_t)b * Skv * ldkv + hh * HD;
  const bf16_t* vp = kp + D;
  const int mykey = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (Sq + KT - 1) / KT;
  const bool ragged = Sq % KT != 0;

  // K and -V fragments of the wave's keys (V negated: dP - Delta is then accumulated as
  // Delta + dO (-V)^T, starting from Delta, which saves a subtraction per score)
  bf16x8 kf[KS], vf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kf[ks] = mykey < Skv ? ld8(kp + (size_t)mykey * ldkv + ks * 16 + 8 * h32) : zero8();
    vf[ks] = neg8(mykey < Skv ? ld8(vp + (size_t)mykey * ldkv + ks * 16 + 8 * h32) : zero8());
  }
  f32x16 dv[DB], dk[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) { zero16(dv[db]); zero16(dk[db]); }

  const __amdgpu_buffer_rsrc_t rq = make_rsrc(q, q_elems * 2u);
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(dO, (uint32_t)((size_t)gridDim.z * Sq * D * 2));
  const __amdgpu_buffer_rsrc_t rl = make_rsrc(lse, (uint32_t)((size_t)gridDim.z * H * Sq * 4));
  const __amdgpu_buffer_rsrc_t rdl = make_rsrc(delta, (uint32_t)((size_t)gridDim.z * H * Sq * 4));
  const uint32_t qbase = (uint32_t)(((size_t)b * Sq * ldq + hh * HD) * 2);
  const uint32_t dbase = (uint32_t)(((size_t)b * Sq * D + hh * HD) * 2);
  const uint32_t lbase = (uint32_t)(((size_t)b * H + hh) * Sq * 4);
  auto load = [&](int t, int s) {
    tile_load<HD, NW>(rq, qbase, (uint32_t)ldq, t * KT, smem + s * 2 * TE);
    tile_load<HD, NW>(rd, dbase, (uint32_t)D, t * KT, smem + s * 2 * TE + TE);
    const uint32_t lo = lbase + (uint32_t)(t * KT + lane) * 4u;
    if (wid == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_ptr_t*)(fsm + s * 2 * KT), 4, lo, 0, 0, 0);
    if (wid == 1) __builtin_amdgcn_raw_ptr_buffer_load_lds(rdl, (lds_ptr_t*)(fsm + s * 2 * KT + KT), 4, lo, 0, 0, 0);
  };
  // S = Q K^T and dP = dO V^T of query unit u: register r holds query srow(r), key l32
  auto s_of = [&](int s, int u, f32x16& sv) {
    const bf16_t* Qs = smem + s * 2 * TE;
    zero16(sv);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) sv = mfma(row_frag<HD>(Qs, u * 32, ks), kf[ks], sv);
  };
  // Delta - dP (= -(dP - Delta)): the accumulator starts from the Delta of the register's query
  // (rows 8 g + 4 h32 .. + 3 for registers 4 g .. 4 g + 3) and adds dO (-V)^T
  auto dp_of = [&](int s, int u, f32x16& dpv) {
    const bf16_t* dOs = smem + s * 2 * TE + TE;
    const float* dls = fsm + s * 2 * KT + KT + u * 32 + 4 * h32;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const float4 d4 = *reinterpret_cast<const float4*>(dls + 8 * g);
      dpv[4 * g] = d4.x; dpv[4 * g + 1] = d4.y; dpv[4 * g + 2] = d4.z; dpv[4 * g + 3] = d4.w;
    }
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) dpv = mfma(row_frag<HD>(dOs, u * 32, ks), vf[ks], dpv);
  };
  // P, dS of the unit (queries past S contribute nothing), then dV^T += dO^T P, dK^T += Q^T dS
  auto grad = [&](int s, int u, const f32x16& sv, int q0, auto rag) {
    f32x16 dpv;
    dp_of(s, u, dpv);
    const float* ls = fsm + s * 2 * KT + u * 32;
    bf16x8 pb[2], sb[2];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int ql = srow(r, h32);
      float p = ex2(fmaf(sv[r], sl2, -ls[ql]));
      float ds = -p * dpv[r];
      if constexpr (decltype(rag)::value) {
        if (q0 + ql >= Sq) { p = 0.f; ds = 0.f; }
      }
      pb[r >> 3][r & 7] = (__bf16)p;
      sb[r >> 3][r & 7] = (__bf16)ds;
    }
    // keep the transposed fragment reads after the arithmetic: hoisted above it they hold
    // registers through the exp2 chain (measured slower)
    __builtin_amdgcn_sched_barrier(0);
    const bf16_t* Qs = smem + s * 2 * TE;
    const bf16_t* dOs = Qs + TE;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        dv[db] = mfma(tr_frag<HD>(dOs, u * 32 + kk * 16, db * 32), pb[kk], dv[db]);
        dk[db] = mfma(tr_frag<HD>(Qs, u * 32 + kk * 16, db * 32), sb[kk], dk[db]);
      }
  };

  load(0, 0);
  if (nt > 1) load(1, 1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  auto tile = [&](int t, auto stg) {
    constexpr int s0 = decltype(stg)::value, s2 = (s0 + 2) % NSTG;
    const bool rag = ragged && t + 1 == nt;
    // head dim 128: one query unit at a time (unrolled, the two units' live ranges spill)
#pragma unroll (HD == 64 ? 2 : 1)
    for (int u = 0; u < 2; ++u) {
      f32x16 sv;
      s_of(s0, u, sv);
      if (rag) grad(s0, u, sv, t * KT + u * 32, std::true_type{});
      else grad(s0, u, sv, t * KT + u * 32, std::false_type{});
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();   // tile t+1 resident; tile t's stage no longer read
    if (t + 2 < nt) load(t + 2, s2);
  };
  int t = 0;
  for (; t + NSTG <= nt; t += NSTG) {
    tile(t, IC<0>{});
    tile(t + 1, IC<1>{});
    tile(t + 2, IC<2>{});
  }
  if (t < nt) tile(t, IC<0>{});
  if (t + 1 < nt) tile(t + 1, IC<1>{});

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  bf16_t* out = dk_out + (size_t)b * Skv * ldo;
  stage_t<HD>(smem, dk, scale, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, out + hh * HD, ldo, id.blk * (32 * NW), Skv);
  __syncthreads();
  stage_t<HD>(smem, dv, 1.0f, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, out + D + hh * HD, ldo, id.blk * (32 * NW), Skv);
}

// ------------------------------------------------------ backward dK, dV at head dim 128: one wave per SIMD
// Four waves of 32 keys (128 keys per workgroup), one per SIMD with the whole register file, the
// work of consecutive 32-query units overlapped inside each wave:
//   unit j:  X_j = [S_j = Q_j K^T, dP_j = dO_j V^T]   (16 MFMAs, VGPR results)
//            V_j = [P_j = exp2(S_j sl2 - lse), dS_j = P_j (dP_j - Delta)]   (vector work)
//            Y_j = [dV^T += dO_j^T P_j, dK^T += Q_j^T dS_j]   (16 MFMAs into AGPR accumulators)
// Step j issues X_{j+1} under V_j, then Y_j.  At head dim 128 a unit has 32 MFMAs (1 024 cycles)
// for about 80 vector instructions, so one wave can issue both; the compiler-scheduled kernel
// keeps its accumulators and operands in AGPRs at this register count and moves the scores back
// and forth through accumulator copies.
// Every MFMA and fragment read is inline assembly with explicit register classes: K, V (B operands
// of X), the Q / dO row fragments (A operands of X) and the accumulators in AGPRs, which gfx950
// MFMAs read and LDS reads write directly (240 AGPRs: K, V 64, accumulators 128, row fragments 48 in a
// ring of twelve slots);
// scores, dP, lse, Delta, P, dS and the transposed fragments (two 8-byte reads form one operand)
// in VGPRs.  The compiler cannot see into the assembly, so the hazards it would cover are covered
// explicitly: s_nop before the vector unit reads MFMA results, before MFMAs read vector results,
// and before the accumulators are read out.
// Each step is 32 regions of one MFMA (and one or two score registers of vector work, split in two
// parts one region apart so that no instruction waits on another of its own region).  Fragment
// reads are issued after the MFMA that last read the register they overwrite (row fragments run
// through a ring of twelve slots: X MFMAs 12..15 reuse the slots of X MFMAs 0..3 of the same unit;
// lse / Delta and the transposed fragments are single-buffered), in a rolling window of at most 15
// in flight; a read is retired about seven regions after it is issued.
// LDS: the Q tiles of the four stages in the first 64 KB, the dO tiles in the next 64 KB (every
// fragment offset fits the instruction's 16-bit offset field), filled two tiles ahead.
namespace dkvh {
constexpr int NST = 4;            // LDS stages
constexpr int NW = 4;             // waves
constexpr int HD = 128;
constexpr int KS = HD / 16;       // MFMA k-steps over the head dimension
constexpr int DB = HD / 32;       // 32-column blocks of the head dimension
constexpr int TE = KT * HD;       // bf16 elements of a 64-row tile
constexpr int TBB = TE * 2;       // bytes of a tile (16 KB)
constexpr int DOFF = NST * TBB;   // byte offset of the dO tiles (64 KB)
constexpr int LPT = 2 * (TE / 512 / NW) + 1;   // buffer loads per wave per tile (Q, dO, lse / Delta / padding)

template <int OFF>
SR_DEV i32x4 rd16a(uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=a"(v) : "v"(a), "i"(OFF));
  return v;
}
template <int OFF>
SR_DEV i32x4 rd16v(uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}
template <int OFF>
SR_DEV i32x2 rdtrv(uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}
// c (VGPR) = a * b (+ c), operands in AGPRs (X)
SR_DEV void mma_v0(f32x16& c, const i32x4& a, const i32x4& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=v"(c) : "a"(a), "a"(b));
}
SR_DEV void mma_v(f32x16& c, const i32x4& a, const i32x4& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "a"(a), "a"(b));
}
// c (AGPR) += a * b, operands in VGPRs (Y)
SR_DEV void mma_a(f32x16& c, const i32x4& a, const i32x4& b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}
template <typename V>
SR_DEV void pin_a(V& v) {
  asm volatile("" : "+a"(v));
}
SR_DEV i32x4 join(const i32x2& lo, const i32x2& hi) {
  i32x4 w;
  w[0] = lo[0]; w[1] = lo[1]; w[2] = hi[0]; w[3] = hi[1];
  return w;
}
// Region schedule of a step (32 regions): the MFMA of region R is X MFMA R (R < 12), Y MFMA R - 12
// of query half 0 (12 <= R < 20), X MFMA R - 8 (20 <= R < 24) or Y MFMA R - 24 of half 1.  X MFMA m:
// k-step m / 2 of S (even m) or of dP (odd m); Y MFMA n: dV^T of column block n / 2 (even
// n) or dK^T (odd n).
constexpr int kind_of(int R) { return R < 12 ? 0 : R < 20 ? 1 : R < 24 ? 0 : 2; }   // 0 X, 1 Y half 0, 2 Y half 1
constexpr int idx_of(int R) { return R < 12 ? R : R < 20 ? R - 12 : R < 24 ? R - 8 : R - 24; }
// region of part a of score register r (part b one region later): registers 0..7 complete before
// region 12, 8..15 before region 20
constexpr int va_region(int r) { return r < 8 ? (r * 3) / 2 : 11 + (r - 8); }
}  // namespace dkvh

__global__ __launch_bounds__(256, 1) void attn_bwd_dkv_h128(const bf16_t* __restrict__ q, int ldq, uint32_t q_elems,
                                                            const bf16_t* __restrict__ kv, int ldkv,
                                                            const bf16_t* __restrict__ dO,
                                                            const float* __restrict__ lse,
                                                            const float* __restrict__ delta,
                                                            bf16_t* __restrict__ dk_out, int ldo, int Sq, int Skv,
                                                            int H, int D, float sl2, float scale) {
  using namespace dkvh;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * NST * TE];   // Q tiles, then dO tiles
  __shared__ __attribute__((aligned(16))) float fsm[NST * 2 * KT];       // stage: lse, Delta of the tile's rows
  __shared__ __attribute__((aligned(16))) float fdummy[64];              // target of the padding loads
  const int lane = threadIdx.x & 63, l32 = lane & 31, h32 = lane >> 5;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const bf16_t* kp = kv + (size_t)b * Skv * ldkv + hh * HD;
  const bf16_t* vp = kp + D;
  const int mykey = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (Sq + KT - 1) / KT;
  const int nu = 2 * nt;   // 32-query units
  const bool ragged = Sq % KT != 0;

  // K and V fragments of the wave's keys, in AGPRs
  i32x4 kf[KS], vf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    kf[ks] = __builtin_bit_cast(i32x4, mykey < Skv ? ld8(kp + (size_t)mykey * ldkv + ks * 16 + 8 * h32) : zero8());
    vf[ks] = __builtin_bit_cast(i32x4, mykey < Skv ? ld8(vp + (size_t)mykey * ldkv + ks * 16 + 8 * h32) : zero8());
  }
  f32x16 dv[DB], dk[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) { zero16(dv[db]); zero16(dk[db]); }
  static_for<KS>([&](auto k) { pin_a(kf[k.value]); pin_a(vf[k.value]); });
  static_for<DB>([&](auto d) { pin_a(dv[d.value]); pin_a(dk[d.value]); });
  asm volatile("s_nop 7" ::: "memory");   // AGPR writes before the first MFMA reads

  const __amdgpu_buffer_rsrc_t rq = make_rsrc(q, q_elems * 2u);
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(dO, (uint32_t)((size_t)gridDim.z * Sq * D * 2));
  const __amdgpu_buffer_rsrc_t rl = make_rsrc(lse, (uint32_t)((size_t)gridDim.z * H * Sq * 4));
  const __amdgpu_buffer_rsrc_t rdl = make_rsrc(delta, (uint32_t)((size_t)gridDim.z * H * Sq * 4));
  const uint32_t qbase = (uint32_t)(((size_t)b * Sq * ldq + hh * HD) * 2);
  const uint32_t dbase = (uint32_t)(((size_t)b * Sq * D + hh * HD) * 2);
  const uint32_t lbase = (uint32_t)(((size_t)b * H + hh) * Sq * 4);
  // tile t into stage s: Q and dO (four 16-byte loads each per wave), lse (wave 0), Delta (wave 1)
  // or a padding load (waves 2, 3: offset past every extent, reads zero, touches no memory), so
  // that every wave has LPT loads per tile in flight
  auto fill = [&](int t, int s) __attribute__((always_inline)) {
    const bool valid = t < nt;
    tile_load<HD, NW>(rq, qbase, (uint32_t)ldq, t * KT, smem + s * TE, valid);
    tile_load<HD, NW>(rd, dbase, (uint32_t)D, t * KT, smem + NST * TE + s * TE, valid);
    const uint32_t lo = valid ? lbase + (uint32_t)(t * KT + lane) * 4u : 0x80000000u;
    if (wid == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_ptr_t*)(fsm + s * 2 * KT), 4, lo, 0, 0, 0);
    else if (wid == 1) __builtin_amdgcn_raw_ptr_buffer_load_lds(rdl, (lds_ptr_t*)(fsm + s * 2 * KT + KT), 4, lo, 0, 0, 0);
    else __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_ptr_t*)fdummy, 4, 0x80000000u, 0, 0, 0);
  };

  // per-lane LDS addresses (stage 0, unit 0 of the Q tiles; the dO tiles DOFF bytes on);
  // stages, units and query halves are instruction offsets
  const uint32_t sbase = lds_addr(smem);
  uint32_t ra[KS], rad[KS];   // row fragments: rows lane % 32 of a unit, k-step ks
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    ra[ks] = sbase + (uint32_t)(l32 * HD + (((2 * ks + h32) ^ swz<HD>(l32)) << 3)) * 2u;
    rad[ks] = ra[ks] + DOFF;
  }
  uint32_t ta[DB][2], tad[DB][2];   // transposed fragments: column block db, first / second read
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int col = 32 * db + 16 * (g & 1) + 4 * (s & 3);
      const int r1 = 4 * (g >> 1) + (s >> 2), r2 = r1 + 8;
      ta[db][0] = sbase + (uint32_t)(r1 * HD + (((col >> 3) ^ swz<HD>(r1)) << 3) + (col & 7)) * 2u;
      ta[db][1] = sbase + (uint32_t)(r2 * HD + (((col >> 3) ^ swz<HD>(r2)) << 3) + (col & 7)) * 2u;
      tad[db][0] = ta[db][0] + DOFF;
      tad[db][1] = ta[db][1] + DOFF;
    }
  }
  const uint32_t la = lds_addr(fsm) + 16u * h32;   // lse / Delta: rows 4 h32 .. + 3 of each group of 8

  // row fragments of X (AGPR): X MFMA m (k-step m / 2 of Q for even m, of dO for odd m) reads slot
  // m % 12
  i32x4 rf[12];
  // transposed fragments of Y (VGPR): a ring of eight pairs, pair n = the A operand of Y MFMA n of
  // either query half (half 1 of a unit is read after half 0's MFMA n, half 0 of the next unit
  // after half 1's)
  i32x2 tf[2 * 2 * DB];
  i32x4 ld[8];                 // lse (groups 0..3), Delta (groups 0..3) of V (VGPR)
  f32x16 sc[2], dpv[2];        // S and dP of a unit, by parity (VGPR)
  bf16x8 pb[2], sb[2];         // P and dS in bf16, query halves (VGPR)
  float pt[16], dt[16];        // part a results of V

  // ---- fragment reads of unit u (U = u % 8: stage (U / 2) % 4, half U % 2)
  // row fragment of X MFMA M (k-step M / 2 of Q for even M, of dO for odd M) into slot M % 12
  auto read_row = [&](auto ui, auto mi) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, M = decltype(mi)::value, K = M / 2;
    constexpr int OFF = ((U / 2) % NST) * TBB + (U % 2) * 32 * HD * 2;
    if constexpr (M % 2 == 0) rf[M % 12] = rd16a<OFF>(ra[K]);
    else rf[M % 12] = rd16a<OFF>(rad[K]);
  };
  // lse (G = 0..3) or Delta (G = 4..7) group G % 4 of unit u
  auto read_stat = [&](auto ui, auto gi) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, G = decltype(gi)::value;
    constexpr int OFF = ((U / 2) % NST) * 2 * KT * 4 + (U % 2) * 32 * 4 + (G >= 4 ? KT * 4 : 0) + (G % 4) * 32;
    ld[G] = rd16v<OFF>(la);
  };
  // transposed fragment pair of Y MFMA N of query half KK into tf[2N], tf[2N+1]: dO^T of column
  // block N / 2 (even N) or Q^T of column block N / 2 (odd N)
  auto read_tr = [&](auto ui, auto kki, auto ni) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, KK = decltype(kki)::value, N = decltype(ni)::value;
    constexpr int C = N / 2;
    constexpr int OFF = ((U / 2) % NST) * TBB + ((U % 2) * 32 + KK * 16) * HD * 2;
    if constexpr (N % 2 == 0) {
      tf[2 * N] = rdtrv<OFF>(tad[C][0]);
      tf[2 * N + 1] = rdtrv<OFF>(tad[C][1]);
    } else {
      tf[2 * N] = rdtrv<OFF>(ta[C][0]);
      tf[2 * N + 1] = rdtrv<OFF>(ta[C][1]);
    }
  };
  // X MFMA M of the unit whose row fragments are in rf, into sc / dpv [P]
  auto xmma = [&](auto pi, auto mi) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, M = decltype(mi)::value, K = M / 2;
    f32x16& acc = M % 2 ? dpv[P] : sc[P];
    const i32x4& fr = rf[M % 12];
    const i32x4& kvf = M % 2 ? vf[K] : kf[K];
    if constexpr (K == 0) mma_v0(acc, fr, kvf);
    else mma_v(acc, fr, kvf);
  };
  // Y MFMA N of query half KK
  auto ymma = [&](auto kki, auto ni) __attribute__((always_inline)) {
    constexpr int KK = decltype(kki)::value, N = decltype(ni)::value, C = N / 2;
    if constexpr (N % 2 == 0)
      mma_a(dv[C], join(tf[2 * N], tf[2 * N + 1]), __builtin_bit_cast(i32x4, pb[KK]));
    else
      mma_a(dk[C], join(tf[2 * N], tf[2 * N + 1]), __builtin_bit_cast(i32x4, sb[KK]));
  };
  // vector work of score register r of the unit in sc / dpv [P] (lse, Delta from ld)
  auto vpart_a = [&](auto pi, auto ri) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, r = decltype(ri)::value;
    pt[r] = ex2(fmaf(sc[P][r], sl2, -__int_as_float(ld[r >> 2][r & 3])));
    dt[r] = dpv[P][r] - __int_as_float(ld[4 + (r >> 2)][r & 3]);
  };
  auto vpart_b = [&](auto ri) __attribute__((always_inline)) {
    constexpr int r = decltype(ri)::value;
    pb[r >> 3][r & 7] = (__bf16)pt[r];
    sb[r >> 3][r & 7] = (__bf16)(pt[r] * dt[r]);
  };
  const int rem = Sq - (nt - 1) * KT;   // valid rows of the last tile
  auto mask_rows = [&](int u) __attribute__((always_inline)) {
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (u * 32 + 8 * g + 4 * h32 + i >= rem) ld[g][i] = 0x7f800000;   // lse = +inf: P = 0, dS = 0
  };

  // reads issued in region R of step j, each after the MFMA that last read the registers it
  // overwrites: rows of X MFMAs 12..15 of unit j+1 (regions 1..4, slots of MFMAs 0..3), of MFMAs
  // 4..11 of unit j+2 (regions 5..12) and of MFMAs 0..3 of unit j+2 (regions 21..24, after X
  // MFMAs 12..15 of unit j+1); transposed pairs of unit j, half 1 (regions 13..20, after half 0's
  // MFMAs) and of unit j+1, half 0 (regions 25..31 and after the last, after half 1's); lse /
  // Delta of unit j+1 (regions 21..24, after the last vector read of unit j's)
  auto reads_of = [&](auto ri, auto ui) __attribute__((always_inline)) {
    constexpr int R = decltype(ri)::value, U = decltype(ui)::value;
    constexpr int UR = (U + 2) % 8, UN = (U + 1) % 8;
    constexpr int mrow = (R >= 1 && R <= 4) ? R + 11 : (R >= 5 && R <= 12) ? R - 1 : (R >= 21 && R <= 24) ? R - 21 : -1;
    constexpr int urow = (R >= 1 && R <= 4) ? UN : UR;
    constexpr int nrow = mrow >= 0 ? 1 : 0;
    constexpr int ntr1 = (R >= 13 && R <= 20) ? R - 13 : -1;   // unit j, half 1
    constexpr int ntr0 = (R >= 25 && R <= 31) ? R - 25 : -1;   // unit j+1, half 0
    constexpr int ntr = (ntr0 >= 0 || ntr1 >= 0) ? 2 : 0;
    // lse / Delta of unit j+1 (the last part-a read of ld is in region va_region(15) = 18): regions 21..24
    constexpr int nst = (R >= 21 && R <= 24) ? 2 : 0;
    constexpr int n = nrow + ntr + nst;
    if constexpr (n > 0) {
      lgkm_wait<15 - n>();
      if constexpr (mrow >= 0) read_row(IC<urow>{}, IC<mrow>{});
      if constexpr (ntr1 >= 0) read_tr(IC<U>{}, IC<1>{}, IC<ntr1>{});
      if constexpr (ntr0 >= 0) read_tr(IC<UN>{}, IC<0>{}, IC<ntr0>{});
      if constexpr (nst > 0) {
        read_stat(IC<UN>{}, IC<2 * (R - 21)>{});
        read_stat(IC<UN>{}, IC<2 * (R - 21) + 1>{});
      }
    }
  };

  auto step = [&](auto ui, int j) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, P = U % 2, Q = 1 - P;
    if constexpr (P == 0) {
      // tile boundary: tile j/2 + 1 resident (only tile j/2 + 2's loads still in flight), then
      // refill the stage of tile j/2 - 1, whose reads all retired during the previous step
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPT) : "memory");
      lds_barrier();
      fill(j / 2 + 3, (U / 2 + 3) % NST);
    }
    lgkm_wait<14>();   // lse / Delta of unit j, rows 0..11 of unit j+1 retired (sixteen reads followed them)
    static_for<8>([&](auto g) { pin(ld[g.value]); });
    if (ragged && j >= nu - 2) mask_rows(P);   // units of the last tile
    asm volatile("s_nop 11" : "+v"(sc[P]), "+v"(dpv[P]));   // X_j's results readable by the vector unit
    __builtin_amdgcn_sched_barrier(0);
    static_for<32>([&](auto ri) {
      constexpr int R = ri.value, KD = kind_of(R), I = idx_of(R);
      if constexpr (R == 12) asm volatile("s_nop 4" : "+v"(pb[0]), "+v"(sb[0]));
      if constexpr (R == 24) asm volatile("s_nop 4" : "+v"(pb[1]), "+v"(sb[1]));
      if constexpr (KD == 0) xmma(IC<Q>{}, IC<I>{});
      else ymma(IC<KD - 1>{}, IC<I>{});
      static_for<16>([&](auto r) {
        if constexpr (va_region(r.value) == R) vpart_a(IC<P>{}, r);
        if constexpr (va_region(r.value) + 1 == R) vpart_b(r);
      });
      reads_of(ri, ui);
      __builtin_amdgcn_sched_barrier(0);
    });
    lgkm_wait<13>();
    read_tr(IC<(U + 1) % 8>{}, IC<0>{}, IC<7>{});
    __builtin_amdgcn_sched_barrier(0);
  };

  // prologue: tiles 0..2 in flight; tile 0 resident; X_0; the reads of step 0
  fill(0, 0);
  fill(1, 1);
  fill(2, 2);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPT) : "memory");
  lds_barrier();
  static_for<12>([&](auto m) {
    if constexpr (m.value == 8) lgkm_wait<7>();
    read_row(IC<0>{}, m);
  });
  lgkm_wait<0>();
  static_for<12>([&](auto m) { xmma(IC<0>{}, m); });
  static_for<4>([&](auto m) { read_row(IC<0>{}, IC<12 + m.value>{}); });   // slots of MFMAs 0..3
  lgkm_wait<0>();
  static_for<4>([&](auto m) { xmma(IC<0>{}, IC<12 + m.value>{}); });
  static_for<12>([&](auto m) {   // rows 0..11 of unit 1, after X_0 read the slots
    if constexpr (m.value % 6 == 0) lgkm_wait<7>();
    read_row(IC<1>{}, m);
  });
  lgkm_wait<7>();
  static_for<8>([&](auto g) { read_stat(IC<0>{}, g); });
  static_for<8>([&](auto n) {
    if constexpr (n.value % 4 == 0) lgkm_wait<7>();
    read_tr(IC<0>{}, IC<0>{}, n);
  });
  __builtin_amdgcn_sched_barrier(0);

  int j = 0;
  for (; j + 8 <= nu; j += 8) {
    step(IC<0>{}, j);
    step(IC<1>{}, j + 1);
    step(IC<2>{}, j + 2);
    step(IC<3>{}, j + 3);
    step(IC<4>{}, j + 4);
    step(IC<5>{}, j + 5);
    step(IC<6>{}, j + 6);
    step(IC<7>{}, j + 7);
  }
  if (j < nu) {   // nu - j is 2, 4 or 6
    step(IC<0>{}, j);
    step(IC<1>{}, j + 1);
    if (j + 2 < nu) {
      step(IC<2>{}, j + 2);
      step(IC<3>{}, j + 3);
      if (j + 4 < nu) {
        step(IC<4>{}, j + 4);
        step(IC<5>{}, j + 5);
      }
    }
  }

  // The last steps read ahead for units past the end: retire those reads with their destination
  // registers still held (pinned behind the wait), or the compiler would hand the registers of
  // reads still in flight to other values.
  lgkm_wait<0>();
  static_for<8>([&](auto g) { pin(ld[g.value]); });
  static_for<12>([&](auto e) { pin_a(rf[e.value]); });
  static_for<4 * DB>([&](auto f) { pin(tf[f.value]); });
  // accumulators readable by the vector unit; every load retired
  static_for<DB>([&](auto d) { pin_a(dv[d.value]); pin_a(dk[d.value]); });
  asm volatile("s_nop 15\n\ts_nop 15" ::: "memory");
  static_for<DB>([&](auto d) { pin_a(dv[d.value]); pin_a(dk[d.value]); });
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  bf16_t* out = dk_out + (size_t)b * Skv * ldo;
  stage_t<HD>(smem, dk, scale, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, out + hh * HD, ldo, id.blk * (32 * NW), Skv);
  __syncthreads();
  stage_t<HD>(smem, dv, 1.0f, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, out + D + hh * HD, ldo, id.blk * (32 * NW), Skv);
}

// ------------------------------------------------------------------------------ backward dQ

// NW waves (32 queries each) per workgroup share the K / V tiles.
template <int HD, int NW>
// Queries: Sq rows of q (stride ldq); keys: Skv rows of kv (stride ldkv, kv_elems addressable
// elements, values D columns on); dQ to dq_out (stride ldo).
__global__ __launch_bounds__(64 * NW, HD == 64 ? 8 / NW : 1) void attn_bwd_dq_mfma(const bf16_t* __restrict__ q, int ldq,
                                                        const bf16_t* __restrict__ kv, int ldkv, uint32_t kv_elems,
                                                        const bf16_t* __restrict__ dO,
                                                        const float* __restrict__ lse, const float* __restrict__ delta,
                                                        bf16_t* __restrict__ dq_out, int ldo, int Sq, int Skv, int H,
                                                        int D, float sl2, float scale) {
  using G = Geo<HD>;
  constexpr int TE = G::TE, TB = G::TB, SGB = G::SGB, KS = G::KS, DB = G::DB;
  __shared__ __attribute__((aligned(16))) bf16_t smem[NSTG * 2 * TE];   // stage: K tile, V tile
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const bf16_t* qp = q + (size_t)b * Sq * ldq + hh * HD;
  const bf16_t* dop = dO + (size_t)b * Sq * D + hh * HD;
  const int myq = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (Skv + KT - 1) / KT;
  const bool ragged = Skv % KT != 0;

  // Q and -dO fragments of the wave's queries (dO negated: dP - Delta is then accumulated as
  // Delta + V (-dO)^T from a constant start, which saves a subtraction per score)
  bf16x8 qf[KS], df[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = myq < Sq ? ld8(qp + (size_t)myq * ldq + ks * 16 + 8 * h32) : zero8();
    df[ks] = neg8(myq < Sq ? ld8(dop + (size_t)myq * D + ks * 16 + 8 * h32) : zero8());
  }
  const float nlse = myq < Sq ? -lse[((size_t)b * H + hh) * Sq + myq] : -INFINITY;
  const float dl_q = myq < Sq ? delta[((size_t)b * H + hh) * Sq + myq] : 0.f;
  f32x16 dl16;   // the dP^T accumulator's start: Delta of the lane's query in every register
#pragma unroll
  for (int r = 0; r < 16; ++r) dl16[r] = dl_q;
  f32x16 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) zero16(dq[db]);

  const __amdgpu_buffer_rsrc_t rq = make_rsrc(kv, kv_elems * 2u);
  const uint32_t kbase = (uint32_t)(((size_t)b * Skv * ldkv + hh * HD) * 2);
  const uint32_t vbase = kbase + (uint32_t)D * 2u;
  RowAddr<HD> ra;
  TrAddr<HD> ta;
  ra.init(lds_addr(smem), lane);
  ta.init(lds_addr(smem), lane);
  constexpr int kLoads = 2 * (G::BLK / NW);   // buffer loads per thread per tile (two tiles)
  auto load = [&](int t, int s) {
    tile_load<HD, NW>(rq, kbase, (uint32_t)ldkv, t * KT, smem + s * 2 * TE, t < nt);
    tile_load<HD, NW>(rq, vbase, (uint32_t)ldkv, t * KT, smem + s * 2 * TE + TE, t < nt);
  };
  // K (tile 0) or V (tile 1) row fragments of key unit U of stage SG
  auto read_rows = [&](auto sg, auto uu, auto tl, RawFrag<true> (&fr)[KS]) {
    constexpr int SG = decltype(sg)::value, U = decltype(uu)::value, TL = decltype(tl)::value;
    static_for<KS>([&](auto ks) { ra.template read<SG * SGB + TL * TB, U * 32, decltype(ks)::value>(fr[ks.value]); });
  };
  // S^T = K Q^T and dP^T = V dO^T of a key unit: register r holds key srow(r), query l32
  auto sd = [&](RawFrag<true> (&kr)[KS], RawFrag<true> (&vr)[KS], f32x16& sv, f32x16& dpv) {
    zero16(sv);
    dpv = dl16;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      sv = mfma(kr[ks].settle(), qf[ks], sv);
      dpv = mfma(vr[ks].settle(), df[ks], dpv);
    }
  };
  // dS^T of unit U (keys past S do not exist), then dQ^T += K^T dS^T (K^T fragments read
  // first, so that their latency hides behind the arithmetic)
  auto grad = [&](auto sg, auto uu, const f32x16& sv, const f32x16& dpv, int k0, auto rag) {
    constexpr int SG = decltype(sg)::value, U = decltype(uu)::value;
    RawFrag<false> fk[DB][2];
    static_for<DB>([&](auto db) {
      static_for<2>([&](auto kk) {
        ta.template read<SG * SGB, U * 32 + decltype(kk)::value * 16, decltype(db)::value>(fk[db.value][kk.value]);
      });
    });
    bf16x8 sb[2];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float p = ex2(fmaf(sv[r], sl2, nlse));
      float ds = -p * dpv[r];
      if constexpr (decltype(rag)::value) {
        if (k0 + srow(r, h32) >= Skv) ds = 0.f;
      }
      sb[r >> 3][r & 7] = (__bf16)ds;
    }
    lgkm_wait<0>();
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) dq[db] = mfma(fk[db][kk].settle(), sb[kk], dq[db]);
  };

  load(0, 0);
  load(1, 1);   // past the last tile: zeros (a uniform count of loads in flight)
  wait_vm_lgkm0<kLoads>();
  lds_barrier();
  auto tile = [&](int t, auto stg) {
    constexpr int s0 = decltype(stg)::value;
    const bool rag = ragged && t + 1 == nt;
    // tile t+2 into the stage of tile t-1, which every wave has left (the barrier that ended
    // tile t-1); it then flies during tiles t and t+1
    load(t + 2, (s0 + 2) % NSTG);
    // both units' S^T / dP^T MFMAs first: unit 1's run while unit 0's arithmetic does
    RawFrag<true> k0r[KS], v0r[KS], k1r[KS], v1r[KS];
    f32x16 sv0, dp0, sv1, dp1;
    read_rows(stg, IC<0>{}, IC<0>{}, k0r);
    read_rows(stg, IC<0>{}, IC<1>{}, v0r);
    lgkm_wait<0>();
    sd(k0r, v0r, sv0, dp0);
    read_rows(stg, IC<1>{}, IC<0>{}, k1r);
    read_rows(stg, IC<1>{}, IC<1>{}, v1r);
    lgkm_wait<0>();
    sd(k1r, v1r, sv1, dp1);
    if (rag) {
      grad(stg, IC<0>{}, sv0, dp0, t * KT, std::true_type{});
      grad(stg, IC<1>{}, sv1, dp1, t * KT + 32, std::true_type{});
    } else {
      grad(stg, IC<0>{}, sv0, dp0, t * KT, std::false_type{});
      grad(stg, IC<1>{}, sv1, dp1, t * KT + 32, std::false_type{});
    }
    wait_vm_lgkm0<kLoads>();   // tile t+1 resident: only tile t+2's loads may still fly
    lds_barrier();             // ... for every wave, and every wave is done with tile t's stage
  };
  int t = 0;
  for (; t + NSTG <= nt; t += NSTG) {
    tile(t, IC<0>{});
    tile(t + 1, IC<1>{});
    tile(t + 2, IC<2>{});
  }
  if (t < nt) tile(t, IC<0>{});
  if (t + 1 < nt) tile(t + 1, IC<1>{});

  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  stage_t<HD>(smem, dq, scale, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, dq_out + (size_t)b * Sq * ldo + hh * HD, ldo, id.blk * (32 * NW), Sq);
}

// ------------------------------------------------------------ backward dQ at head dim 128: one wave per SIMD
// The register-explicit form of the dK/dV kernel above, for dQ: four waves of 32 queries, one per
// SIMD, streaming 64-key tiles (two 32-key units each):
//   unit j:  X_j = [S^T_j = K_j Q^T, Delta - dP^T_j = Delta + V_j (-dO)^T]   (16 MFMAs, VGPR results)
//            V_j = [P = exp2(S^T sl2 - lse), dS^T = -P (Delta - dP^T)]   (lse, Delta: the lane's query)
//            Y_j = [dQ^T += K_j^T dS^T_j]   (8 MFMAs into AGPR accumulators)
// Q and -dO of the wave's queries (B operands of X), the accumulators and the K / V row fragments
// (A operands of X, a ring of twelve slots) in AGPRs; scores, dP, P, dS and the transposed K
// fragments (a ring of eight pairs) in VGPRs.  24 one-MFMA regions per step, vector work split in
// two parts one region apart, fragment reads in a rolling window of at most 15 in flight, each
// issued after the MFMA that last read the registers it overwrites.  LDS: the K tiles of the four
// stages in the first 64 KB, the V tiles in the next 64 KB, filled two tiles ahead.
namespace dqh {
constexpr int NST = 4;
constexpr int NW = 4;
constexpr int HD = 128;
constexpr int KS = HD / 16;
constexpr int DB = HD / 32;
constexpr int TE = KT * HD;
constexpr int TBB = TE * 2;
constexpr int VOFF = NST * TBB;                // byte offset of the V tiles (64 KB)
constexpr int LPT = 2 * (TE / 512 / NW);       // buffer loads per wave per tile (K, V)
// region R of a step: X MFMA R (R < 12), Y MFMA R - 12 (12 <= R < 16, query half... key half 0),
// X MFMA R - 4 (16 <= R < 20), Y MFMA R - 16 (20 <= R < 24, key half 1).  X MFMA m: k-step m / 2 of
// S^T (even m) or of Delta - dP^T (odd m); Y MFMA n: key half n / 4, column block n % 4.
constexpr int kind_of(int R) { return R < 12 ? 0 : R < 16 ? 1 : R < 20 ? 0 : 1; }
constexpr int idx_of(int R) { return R < 12 ? R : R < 16 ? R - 12 : R < 20 ? R - 4 : R - 16; }
constexpr int va_region(int r) { return r < 8 ? (r * 3) / 2 : 11 + (r - 8); }
}  // namespace dqh

__global__ __launch_bounds__(256, 1) void attn_bwd_dq_h128(const bf16_t* __restrict__ q, int ldq,
                                                           const bf16_t* __restrict__ kv, int ldkv,
                                                           uint32_t kv_elems, const bf16_t* __restrict__ dO,
                                                           const float* __restrict__ lse,
                                                           const float* __restrict__ delta,
                                                           bf16_t* __restrict__ dq_out, int ldo, int Sq, int Skv,
                                                           int H, int D, float sl2, float scale) {
  using namespace dqh;
  using dkvh::rd16a;
  using dkvh::rdtrv;
  using dkvh::mma_v0;
  using dkvh::mma_v;
  using dkvh::mma_a;
  using dkvh::pin_a;
  using dkvh::join;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * NST * TE];   // K tiles, then V tiles
  const int lane = threadIdx.x & 63, l32 = lane & 31, h32 = lane >> 5;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const bf16_t* qp = q + (size_t)b * Sq * ldq + hh * HD;
  const bf16_t* dop = dO + (size_t)b * Sq * D + hh * HD;
  const int myq = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (Skv + KT - 1) / KT;
  const int nu = 2 * nt;
  const bool ragged = Skv % KT != 0;

  // Q and -dO fragments of the wave's queries (AGPR); dO negated so that the dP^T chain
  // accumulates Delta - dP^T from a start tuple holding the query's Delta
  i32x4 qf[KS], df[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    qf[ks] = __builtin_bit_cast(i32x4, myq < Sq ? ld8(qp + (size_t)myq * ldq + ks * 16 + 8 * h32) : zero8());
    df[ks] = __builtin_bit_cast(i32x4, neg8(myq < Sq ? ld8(dop + (size_t)myq * D + ks * 16 + 8 * h32) : zero8()));
  }
  const float nlse = myq < Sq ? -lse[((size_t)b * H + hh) * Sq + myq] : -INFINITY;
  const float dl_q = myq < Sq ? delta[((size_t)b * H + hh) * Sq + myq] : 0.f;
  f32x16 dl16;
#pragma unroll
  for (int r = 0; r < 16; ++r) dl16[r] = dl_q;
  f32x16 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) zero16(dq[db]);
  static_for<KS>([&](auto k) { pin_a(qf[k.value]); pin_a(df[k.value]); });
  static_for<DB>([&](auto d) { pin_a(dq[d.value]); });
  asm volatile("s_nop 7" ::: "memory");   // AGPR writes before the first MFMA reads

  const __amdgpu_buffer_rsrc_t rkv = make_rsrc(kv, kv_elems * 2u);
  const uint32_t kbase = (uint32_t)(((size_t)b * Skv * ldkv + hh * HD) * 2);
  const uint32_t vbase = kbase + (uint32_t)D * 2u;
  auto fill = [&](int t, int s) __attribute__((always_inline)) {
    const bool valid = t < nt;
    tile_load<HD, NW>(rkv, kbase, (uint32_t)ldkv, t * KT, smem + s * TE, valid);
    tile_load<HD, NW>(rkv, vbase, (uint32_t)ldkv, t * KT, smem + NST * TE + s * TE, valid);
  };

  const uint32_t sbase = lds_addr(smem);
  uint32_t ra[KS], rav[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    ra[ks] = sbase + (uint32_t)(l32 * HD + (((2 * ks + h32) ^ swz<HD>(l32)) << 3)) * 2u;
    rav[ks] = ra[ks] + VOFF;
  }
  uint32_t ta[DB][2];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int col = 32 * db + 16 * (g & 1) + 4 * (s & 3);
      const int r1 = 4 * (g >> 1) + (s >> 2), r2 = r1 + 8;
      ta[db][0] = sbase + (uint32_t)(r1 * HD + (((col >> 3) ^ swz<HD>(r1)) << 3) + (col & 7)) * 2u;
      ta[db][1] = sbase + (uint32_t)(r2 * HD + (((col >> 3) ^ swz<HD>(r2)) << 3) + (col & 7)) * 2u;
    }
  }

  i32x4 rf[12];                // K / V row fragments of X, slot m % 12 (AGPR)
  i32x2 tf[2 * 2 * DB];        // K^T fragments of Y MFMA n: tf[2n], tf[2n+1] (VGPR)
  f32x16 sc[2], dpv[2];        // S^T and Delta - dP^T of a unit, by parity (VGPR)
  bf16x8 sb[2];                // dS^T in bf16, key halves (VGPR)
  float pt[16], dt[16];

  // row fragment of X MFMA M of unit u (K k-step M / 2 for even M, V for odd M) into slot M % 12
  auto read_row = [&](auto ui, auto mi) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, M = decltype(mi)::value, K = M / 2;
    constexpr int OFF = ((U / 2) % NST) * TBB + (U % 2) * 32 * HD * 2;
    if constexpr (M % 2 == 0) rf[M % 12] = rd16a<OFF>(ra[K]);
    else rf[M % 12] = rd16a<OFF>(rav[K]);
  };
  // K^T fragment pair of Y MFMA N (key half N / 4, column block N % 4) of unit u
  auto read_tr = [&](auto ui, auto ni) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, N = decltype(ni)::value, KK = N / 4, C = N % 4;
    constexpr int OFF = ((U / 2) % NST) * TBB + ((U % 2) * 32 + KK * 16) * HD * 2;
    tf[2 * N] = rdtrv<OFF>(ta[C][0]);
    tf[2 * N + 1] = rdtrv<OFF>(ta[C][1]);
  };
  auto xmma = [&](auto pi, auto mi) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, M = decltype(mi)::value, K = M / 2;
    if constexpr (M % 2 == 0) {
      if constexpr (K == 0) mma_v0(sc[P], rf[0], qf[0]);
      else mma_v(sc[P], rf[M % 12], qf[K]);
    } else {
      if constexpr (K == 0) asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %3" : "=v"(dpv[P]) : "a"(rf[1]), "a"(df[0]), "v"(dl16));
      else mma_v(dpv[P], rf[M % 12], df[K]);
    }
  };
  auto ymma = [&](auto ni) __attribute__((always_inline)) {
    constexpr int N = decltype(ni)::value, KK = N / 4, C = N % 4;
    mma_a(dq[C], join(tf[2 * N], tf[2 * N + 1]), __builtin_bit_cast(i32x4, sb[KK]));
  };
  auto vpart_a = [&](auto pi, auto ri) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, r = decltype(ri)::value;
    pt[r] = ex2(fmaf(sc[P][r], sl2, nlse));
    dt[r] = dpv[P][r];
  };
  auto vpart_b = [&](auto ri) __attribute__((always_inline)) {
    constexpr int r = decltype(ri)::value;
    sb[r >> 3][r & 7] = (__bf16)(-pt[r] * dt[r]);
  };
  const int rem = Skv - (nt - 1) * KT;   // valid keys of the last tile
  // keys past Skv (units of the last, ragged tile): S^T = -inf, so P = 0 and dS = 0
  auto mask_keys = [&](auto pi, int u) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (u * 32 + srow(r, h32) >= rem) sc[P][r] = -INFINITY;
  };
  // reads issued in region R of step j: rows of X MFMAs 12..15 of unit j+1 (regions 1..4, slots of
  // MFMAs 0..3), of MFMAs 4..11 of unit j+2 (regions 5..12), of MFMAs 0..3 of unit j+2 (regions
  // 17..20, after X MFMAs 12..15 of unit j+1); the K^T pair of Y MFMA n of unit j+1 after Y MFMA n
  // of unit j (regions 13..16 for n = 0..3, 21..23 and after the last for n = 4..7)
  auto reads_of = [&](auto ri, auto ui) __attribute__((always_inline)) {
    constexpr int R = decltype(ri)::value, U = decltype(ui)::value;
    constexpr int UR = (U + 2) % 8, UN = (U + 1) % 8;
    constexpr int mrow = (R >= 1 && R <= 4) ? R + 11 : (R >= 5 && R <= 12) ? R - 1 : (R >= 17 && R <= 20) ? R - 17 : -1;
    constexpr int urow = (R >= 1 && R <= 4) ? UN : UR;
    constexpr int ntr = (R >= 13 && R <= 16) ? R - 13 : (R >= 21 && R <= 23) ? R - 17 : -1;
    constexpr int n = (mrow >= 0 ? 1 : 0) + (ntr >= 0 ? 2 : 0);
    if constexpr (n > 0) {
      lgkm_wait<15 - n>();
      if constexpr (mrow >= 0) read_row(IC<urow>{}, IC<mrow>{});
      if constexpr (ntr >= 0) read_tr(IC<UN>{}, IC<ntr>{});
    }
  };

  auto step = [&](auto ui, int j) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, P = U % 2, Q = 1 - P;
    if constexpr (P == 0) {
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(LPT) : "memory");
      lds_barrier();
      fill(j / 2 + 3, (U / 2 + 3) % NST);
    }
    // rows of X MFMAs 0..3 of unit j+1 retired: they were read in regions 17..20 of the previous
    // step, and eight reads followed them
    lgkm_wait<8>();
    asm volatile("s_nop 11" : "+v"(sc[P]), "+v"(dpv[P]));   // X_j's results readable by the vector unit
    if (ragged && j >= nu - 2) mask_keys(IC<P>{}, P);
    __builtin_amdgcn_sched_barrier(0);
    static_for<24>([&](auto ri) {
      constexpr int R = ri.value, KD = kind_of(R), I = idx_of(R);
      if constexpr (R == 12) asm volatile("s_nop 4" : "+v"(sb[0]));
      if constexpr (R == 20) asm volatile("s_nop 4" : "+v"(sb[1]));
      if constexpr (KD == 0) xmma(IC<Q>{}, IC<I>{});
      else ymma(IC<I>{});
      static_for<16>([&](auto r) {
        if constexpr (va_region(r.value) == R) vpart_a(IC<P>{}, r);
        if constexpr (va_region(r.value) + 1 == R) vpart_b(r);
      });
      reads_of(ri, ui);
      __builtin_amdgcn_sched_barrier(0);
    });
    lgkm_wait<13>();
    read_tr(IC<(U + 1) % 8>{}, IC<7>{});
    __builtin_amdgcn_sched_barrier(0);
  };

  fill(0, 0);
  fill(1, 1);
  fill(2, 2);
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * LPT) : "memory");
  lds_barrier();
  static_for<12>([&](auto m) {
    if constexpr (m.value == 8) lgkm_wait<7>();
    read_row(IC<0>{}, m);
  });
  lgkm_wait<0>();
  static_for<12>([&](auto m) { xmma(IC<0>{}, m); });
  static_for<4>([&](auto m) { read_row(IC<0>{}, IC<12 + m.value>{}); });
  lgkm_wait<0>();
  static_for<4>([&](auto m) { xmma(IC<0>{}, IC<12 + m.value>{}); });
  static_for<12>([&](auto m) {
    if constexpr (m.value % 6 == 0) lgkm_wait<7>();
    read_row(IC<1>{}, m);
  });
  static_for<8>([&](auto n) {
    if constexpr (n.value % 4 == 0) lgkm_wait<7>();
    read_tr(IC<0>{}, n);
  });
  __builtin_amdgcn_sched_barrier(0);

  int j = 0;
  for (; j + 8 <= nu; j += 8) {
    step(IC<0>{}, j);
    step(IC<1>{}, j + 1);
    step(IC<2>{}, j + 2);
    step(IC<3>{}, j + 3);
    step(IC<4>{}, j + 4);
    step(IC<5>{}, j + 5);
    step(IC<6>{}, j + 6);
    step(IC<7>{}, j + 7);
  }
  if (j < nu) {
    step(IC<0>{}, j);
    step(IC<1>{}, j + 1);
    if (j + 2 < nu) {
      step(IC<2>{}, j + 2);
      step(IC<3>{}, j + 3);
      if (j + 4 < nu) {
        step(IC<4>{}, j + 4);
        step(IC<5>{}, j + 5);
      }
    }
  }

  lgkm_wait<0>();
  static_for<12>([&](auto e) { pin_a(rf[e.value]); });
  static_for<4 * DB>([&](auto f) { pin(tf[f.value]); });
  static_for<DB>([&](auto d) { pin_a(dq[d.value]); });
  asm volatile("s_nop 15\n\ts_nop 15" ::: "memory");
  static_for<DB>([&](auto d) { pin_a(dq[d.value]); });
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  stage_t<HD>(smem, dq, scale, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, dq_out + (size_t)b * Sq * ldo + hh * HD, ldo, id.blk * (32 * NW), Sq);
}

// ------------------------------------------------------------ forward at head dim 128: one wave per SIMD
// The register-explicit form of the attention forward: four waves of 32 queries, one per SIMD,
// streaming 64-key tiles, one tile per step:
//   X_t = [S^T_t = K_t Q^T]   (16 MFMAs: two 32-key units x 8 k-steps, VGPR results)
//   V_t = [row max, lazy rescale, P^T = exp2(S^T sl2 - m) in bf16]   (vector work)
//   Y_t = [l += colsums(P^T) (4 MFMAs with a ones operand), O^T += V_t^T P^T (16 MFMAs)]
// Step t issues X_{t+1} under V_t, then Y_t.  Q of the wave's queries (B operand of X), the O^T
// and row-sum accumulators, the ones operand and the K row fragments (A operands of X, a ring of
// twelve slots) in AGPRs; scores, P and the V^T fragments (a ring of eight pairs) in VGPRs.  36
// one-MFMA regions per step, fragment reads in a rolling window of at most 15 in flight, each
// issued after the MFMA that last read the registers it overwrites.  A step reads fragments of
// tiles t+1 and t+2, so the tile barrier waits for every fill (tile t+2's, issued a step
// earlier).  LDS: K tiles of the four stages in the first 64 KB, V tiles in the next 64 KB.
namespace fwh {
constexpr int NST = 4;
constexpr int NW = 4;
constexpr int HD = 128;
constexpr int KS = HD / 16;
constexpr int DB = HD / 32;
constexpr int TE = KT * HD;
constexpr int TBB = TE * 2;
constexpr int VOFF = NST * TBB;
// region R: X MFMA R (R < 16: unit R % 2, k-step R / 2); Y MFMA R - 16 of unit 0 (16 <= R < 26)
// or R - 26 of unit 1: Y MFMA i < 2 is the row-sum MFMA of query half... key half i, i >= 2 the
// O^T MFMA of column block (i - 2) / 2, key half (i - 2) % 2.
// part a (exp) of score register r of unit u in region 5 + 8 u + r / 2, part b one region later
}  // namespace fwh

__global__ __launch_bounds__(256, 1) void attn_fwd_h128(const bf16_t* __restrict__ q, int ldq,
                                                        const bf16_t* __restrict__ kv, int ldkv, uint32_t kv_elems,
                                                        bf16_t* __restrict__ O, float* __restrict__ lse, int Sq,
                                                        int Skv, int H, int D, float sl2) {
  using namespace fwh;
  using dkvh::rd16a;
  using dkvh::rdtrv;
  using dkvh::mma_v0;
  using dkvh::mma_v;
  using dkvh::mma_a;
  using dkvh::pin_a;
  using dkvh::join;
  __shared__ __attribute__((aligned(1024))) bf16_t smem[2 * NST * TE];   // K tiles, then V tiles
  const int lane = threadIdx.x & 63, l32 = lane & 31, h32 = lane >> 5;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const bf16_t* qp = q + (size_t)b * Sq * ldq + hh * HD;
  const int myq = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (Skv + KT - 1) / KT;
  const bool ragged = Skv % KT != 0;

  i32x4 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qf[ks] = __builtin_bit_cast(i32x4, myq < Sq ? ld8(qp + (size_t)myq * ldq + ks * 16 + 8 * h32) : zero8());
  f32x16 o[DB], lsum;
#pragma unroll
  for (int db = 0; db < DB; ++db) zero16(o[db]);
  zero16(lsum);
  // softmax denominators on the matrix cores: an A operand whose row 0 is all ones turns the P^T
  // MFMA into the column sums of P^T, so lsum[0] of lane l32 (first half) sums the bf16
  // probabilities of query l32 (the values the PV product uses); every other element stays zero
  bf16x8 ones8;
#pragma unroll
  for (int i = 0; i < 8; ++i) ones8[i] = (__bf16)(l32 == 0 ? 1.0f : 0.0f);
  i32x4 ones = __builtin_bit_cast(i32x4, ones8);
  static_for<KS>([&](auto k) { pin_a(qf[k.value]); });
  static_for<DB>([&](auto d) { pin_a(o[d.value]); });
  pin_a(lsum);
  pin_a(ones);
  asm volatile("s_nop 7" ::: "memory");
  float m_run = -INFINITY;   // running reference max of the raw scores

  const __amdgpu_buffer_rsrc_t rkv = make_rsrc(kv, kv_elems * 2u);
  const uint32_t kbase = (uint32_t)(((size_t)b * Skv * ldkv + hh * HD) * 2);
  const uint32_t vbase = kbase + (uint32_t)D * 2u;
  auto fill = [&](int t, int s) __attribute__((always_inline)) {
    const bool valid = t < nt;
    tile_load<HD, NW>(rkv, kbase, (uint32_t)ldkv, t * KT, smem + s * TE, valid);
    tile_load<HD, NW>(rkv, vbase, (uint32_t)ldkv, t * KT, smem + NST * TE + s * TE, valid);
  };
  const uint32_t sbase = lds_addr(smem);
  uint32_t ra[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) ra[ks] = sbase + (uint32_t)(l32 * HD + (((2 * ks + h32) ^ swz<HD>(l32)) << 3)) * 2u;
  uint32_t tav[DB][2];
  {
    const int g = lane >> 4, s = lane & 15;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int col = 32 * db + 16 * (g & 1) + 4 * (s & 3);
      const int r1 = 4 * (g >> 1) + (s >> 2), r2 = r1 + 8;
      tav[db][0] = sbase + VOFF + (uint32_t)(r1 * HD + (((col >> 3) ^ swz<HD>(r1)) << 3) + (col & 7)) * 2u;
      tav[db][1] = sbase + VOFF + (uint32_t)(r2 * HD + (((col >> 3) ^ swz<HD>(r2)) << 3) + (col & 7)) * 2u;
    }
  }

  i32x4 rf[12];             // K row fragments of X, slot m % 12 (AGPR)
  i32x2 tf[16];             // V^T fragments of O^T MFMA n (n = 0..7 of a unit): tf[2n], tf[2n+1] (VGPR)
  f32x16 sc[2][2];          // S^T of the two units of a tile, by parity (VGPR)
  bf16x8 pb[2][2];          // P^T in bf16: unit, key half (VGPR)
  float pt[2][16];

  // K row fragment of X MFMA M of tile t (T = t % 4): unit M % 2, k-step M / 2, slot M % 12
  auto read_row = [&](auto ti, auto mi) __attribute__((always_inline)) {
    constexpr int T = decltype(ti)::value, M = decltype(mi)::value;
    constexpr int OFF = (T % NST) * TBB + (M % 2) * 32 * HD * 2;
    rf[M % 12] = rd16a<OFF>(ra[M / 2]);
  };
  // V^T pair of O^T MFMA N (column block N / 2, key half N % 2) of unit U of tile t
  auto read_tr = [&](auto ti, auto ui, auto ni) __attribute__((always_inline)) {
    constexpr int T = decltype(ti)::value, U = decltype(ui)::value, N = decltype(ni)::value;
    constexpr int C = N / 2, KK = N % 2;
    constexpr int OFF = (T % NST) * TBB + (U * 32 + KK * 16) * HD * 2;
    tf[2 * N] = rdtrv<OFF>(tav[C][0]);
    tf[2 * N + 1] = rdtrv<OFF>(tav[C][1]);
  };
  auto xmma = [&](auto pi, auto mi) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, M = decltype(mi)::value, U = M % 2, K = M / 2;
    if constexpr (K == 0) mma_v0(sc[P][U], rf[M % 12], qf[0]);
    else mma_v(sc[P][U], rf[M % 12], qf[K]);
  };
  // Y MFMA I of unit U: I < 2 row sums of key half I, else O^T of column block (I-2)/2, key half (I-2)%2
  auto ymma = [&](auto ui, auto ii) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, I = decltype(ii)::value;
    if constexpr (I < 2) {
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(lsum) : "a"(ones), "v"(__builtin_bit_cast(i32x4, pb[U][I])));
    } else {
      constexpr int N = I - 2, C = N / 2, KK = N % 2;
      mma_a(o[C], join(tf[2 * N], tf[2 * N + 1]), __builtin_bit_cast(i32x4, pb[U][KK]));
    }
  };
  const int rem = Skv - (nt - 1) * KT;
  auto mask_keys = [&](auto pi) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value;
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (u * 32 + srow(r, h32) >= rem) sc[P][u][r] = -INFINITY;
  };
  float nm = 0.f;
  // row max of the tile over registers R0 .. R0+7 of both units (regions 0..3), the reference update
  // (region 4)
  float mx = -INFINITY;
  auto vmax = [&](auto pi, auto qi) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, Qp = decltype(qi)::value;
    static_for<8>([&](auto i) {
      constexpr int r = (Qp % 2) * 8 + i.value, u = Qp / 2;
      mx = fmaxf(mx, sc[P][u][r]);
    });
  };
  auto vref = [&]() __attribute__((always_inline)) {
    mx = half_pair_max(mx);
    // lazy rescaling: the reference max m_run moves (and O, l are rescaled) only when a row's
    // max has grown by more than 8 in exp2 units; otherwise p = 2^((s - m_run) c) <= 256
    const float grow = (fmaxf(m_run, mx) - m_run) * sl2;   // +inf on the first tile
    if (__ballot(grow > 8.0f)) {
      const float m_ref = grow > 8.0f ? mx : m_run;
      const float alpha = ex2((m_run - m_ref) * sl2);
      asm volatile("s_nop 15\n\ts_nop 3" ::: "memory");   // the accumulators' last MFMA writes landed
      static_for<DB>([&](auto d) { pin_a(o[d.value]); });
      pin_a(lsum);
      lsum[0] *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      static_for<DB>([&](auto d) { pin_a(o[d.value]); });
      pin_a(lsum);
      asm volatile("s_nop 4" ::: "memory");   // accumulator writes before the next MFMAs read them
      m_run = m_ref;
    }
    nm = -m_run * sl2;
    mx = -INFINITY;
  };
  auto vpart_a = [&](auto pi, auto ui, auto ri) __attribute__((always_inline)) {
    constexpr int P = decltype(pi)::value, U = decltype(ui)::value, r = decltype(ri)::value;
    pt[U][r] = ex2(fmaf(sc[P][U][r], sl2, nm));
  };
  auto vpart_b = [&](auto ui, auto ri) __attribute__((always_inline)) {
    constexpr int U = decltype(ui)::value, r = decltype(ri)::value;
    pb[U][r >> 3][r & 7] = (__bf16)pt[U][r];
  };
  // reads issued in region R of step t: K rows of X MFMAs 12..15 of tile t+1 (regions 1..4, slots
  // of MFMAs 0..3), of MFMAs 4..11 of tile t+2 (regions 5..12), of MFMAs 0..3 of tile t+2 (regions
  // 13..16, after X MFMAs 12..15); V^T pairs of unit 1 of tile t after unit 0's O^T MFMA n (regions
  // 19..26) and of unit 0 of tile t+1 after unit 1's (regions 29..35 and after the last)
  auto reads_of = [&](auto ri, auto ti) __attribute__((always_inline)) {
    constexpr int R = decltype(ri)::value, T = decltype(ti)::value;
    constexpr int mrow = (R >= 1 && R <= 4) ? R + 11 : (R >= 5 && R <= 12) ? R - 1 : (R >= 13 && R <= 16) ? R - 13 : -1;
    constexpr int trow = (R >= 1 && R <= 4) ? (T + 1) % 4 : (T + 2) % 4;
    constexpr int ntr1 = (R >= 19 && R <= 26) ? R - 19 : -1;   // unit 1 of tile t
    constexpr int ntr0 = (R >= 29 && R <= 35) ? R - 29 : -1;   // unit 0 of tile t+1
    constexpr int n = (mrow >= 0 ? 1 : 0) + (ntr1 >= 0 || ntr0 >= 0 ? 2 : 0);
    if constexpr (n > 0) {
      lgkm_wait<15 - n>();
      if constexpr (mrow >= 0) read_row(IC<trow>{}, IC<mrow>{});
      if constexpr (ntr1 >= 0) read_tr(IC<T>{}, IC<1>{}, IC<ntr1>{});
      if constexpr (ntr0 >= 0) read_tr(IC<(T + 1) % 4>{}, IC<0>{}, IC<ntr0>{});
    }
  };

  auto step = [&](auto ti, int t) __attribute__((always_inline)) {
    constexpr int T = decltype(ti)::value, P = T % 2, Q = 1 - P;
    // tile barrier: tiles t+1, t+2 resident (tile t+2's fill was the last issued), then refill
    // the stage of tile t-1, whose reads all retired during the previous step
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    lds_barrier();
    fill(t + 3, (T + 3) % NST);
    lgkm_wait<13>();
    asm volatile("s_nop 11" : "+v"(sc[P][0]), "+v"(sc[P][1]));   // X_t's results readable by the vector unit
    if (ragged && t == nt - 1) mask_keys(IC<P>{});
    __builtin_amdgcn_sched_barrier(0);
    static_for<36>([&](auto ri) {
      constexpr int R = ri.value;
      if constexpr (R == 16) asm volatile("s_nop 4" : "+v"(pb[0][0]), "+v"(pb[0][1]));
      if constexpr (R == 26) asm volatile("s_nop 4" : "+v"(pb[1][0]), "+v"(pb[1][1]));
      // consumers whose reads are fewer than fifteen reads back: X MFMAs 12..15 (slots refilled in
      // regions 1..4, ten reads before) and the O^T MFMAs of unit 1 (pairs read in regions 19..26,
      // twelve or more reads before)
      if constexpr (R >= 12 && R <= 15) lgkm_wait<10>();
      if constexpr (R >= 28) lgkm_wait<12>();
      if constexpr (R < 16) xmma(IC<Q>{}, IC<R>{});
      else if constexpr (R < 26) ymma(IC<0>{}, IC<R - 16>{});
      else ymma(IC<1>{}, IC<R - 26>{});
      if constexpr (R < 4) vmax(IC<P>{}, IC<R>{});
      if constexpr (R == 4) vref();
      static_for<16>([&](auto r) {
        constexpr int ra0 = 5 + r.value / 2, ra1 = 13 + r.value / 2;
        if constexpr (ra0 == R) vpart_a(IC<P>{}, IC<0>{}, r);
        if constexpr (ra0 + 1 == R) vpart_b(IC<0>{}, r);
        if constexpr (ra1 == R) vpart_a(IC<P>{}, IC<1>{}, r);
        if constexpr (ra1 + 1 == R) vpart_b(IC<1>{}, r);
      });
      reads_of(ri, ti);
      __builtin_amdgcn_sched_barrier(0);
    });
    lgkm_wait<13>();
    read_tr(IC<(T + 1) % 4>{}, IC<0>{}, IC<7>{});
    __builtin_amdgcn_sched_barrier(0);
  };

  // prologue: tiles 0..2 resident; X_0; the reads of step 0 (rows 0..11 of tile 1, V^T of tile 0 unit 0)
  fill(0, 0);
  fill(1, 1);
  fill(2, 2);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  lds_barrier();
  static_for<12>([&](auto m) {
    if constexpr (m.value == 8) lgkm_wait<7>();
    read_row(IC<0>{}, m);
  });
  lgkm_wait<0>();
  static_for<12>([&](auto m) { xmma(IC<0>{}, m); });
  static_for<4>([&](auto m) { read_row(IC<0>{}, IC<12 + m.value>{}); });
  lgkm_wait<0>();
  static_for<4>([&](auto m) { xmma(IC<0>{}, IC<12 + m.value>{}); });
  static_for<12>([&](auto m) {
    if constexpr (m.value % 6 == 0) lgkm_wait<7>();
    read_row(IC<1>{}, m);
  });
  static_for<8>([&](auto n) {
    if constexpr (n.value % 4 == 0) lgkm_wait<7>();
    read_tr(IC<0>{}, IC<0>{}, n);
  });
  __builtin_amdgcn_sched_barrier(0);

  int t = 0;
  for (; t + 4 <= nt; t += 4) {
    step(IC<0>{}, t);
    step(IC<1>{}, t + 1);
    step(IC<2>{}, t + 2);
    step(IC<3>{}, t + 3);
  }
  if (t < nt) {
    step(IC<0>{}, t);
    if (t + 1 < nt) {
      step(IC<1>{}, t + 1);
      if (t + 2 < nt) step(IC<2>{}, t + 2);
    }
  }

  lgkm_wait<0>();
  static_for<12>([&](auto e) { pin_a(rf[e.value]); });
  static_for<16>([&](auto f) { pin(tf[f.value]); });
  static_for<DB>([&](auto d) { pin_a(o[d.value]); });
  pin_a(lsum);
  asm volatile("s_nop 15\n\ts_nop 15" ::: "memory");
  static_for<DB>([&](auto d) { pin_a(o[d.value]); });
  pin_a(lsum);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();   // every wave is done with the stages before they hold the output
  const float l_tot = half_pair_sum(lsum[0]);   // the second half's element is zero
  if (h32 == 0 && myq < Sq) lse[((size_t)b * H + hh) * Sq + myq] = m_run * sl2 + log2f(l_tot);
  stage_t<HD>(smem, o, 1.0f / l_tot, wid, lane);
  __syncthreads();
  unstage<HD, NW>(smem, O + (size_t)b * Sq * D + hh * HD, D, id.blk * (32 * NW), Sq);
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

// ------------------------------------------------------------------------- column sums
// colsum[b,h,j] = sum over the S queries i of P[i,j], P = exp2(s * sl2 - lse) the forward's
// probabilities: the attention token j receives in head h.  MFMA: the dK/dV kernel's score
// half; a wave owns 32 keys (key per lane) and streams 64-query tiles; each lane sums its
// 16 query rows per unit in tile, unit and row order, then the two half-waves (which hold
// the other 16 rows of each unit) are added.  Deterministic.
template <int NW>
__global__ __launch_bounds__(64 * NW, 8 / NW) void attn_colsum_mfma(const bf16_t* __restrict__ qkv,
                                                           const float* __restrict__ lse,
                                                           float* __restrict__ colsum, int S, int H, int D,
                                                           float sl2) {
  constexpr int HD = 64;   // the deterministic model's head dim (the selector's block)
  constexpr int TE = Geo<HD>::TE;
  __shared__ __attribute__((aligned(16))) bf16_t smem[NSTG * TE];   // stage: Q tile
  __shared__ __attribute__((aligned(16))) float fsm[NSTG * KT];     // stage: lse of the tile's rows
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, l32 = lane & 31, h32 = lane >> 5;
  const TileId id = xcd_tile_id();
  const int b = id.b, hh = id.h;
  const size_t ld = 3 * (size_t)D;
  const bf16_t* kp = qkv + (size_t)b * S * ld + D + hh * HD;
  const int mykey = id.blk * (32 * NW) + wid * 32 + l32;
  const int nt = (S + KT - 1) / KT;
  const bool ragged = S % KT != 0;

  bf16x8 kf[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) kf[ks] = mykey < S ? ld8(kp + (size_t)mykey * ld + ks * 16 + 8 * h32) : zero8();

  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qkv, (uint32_t)((size_t)gridDim.z * S * ld * 2));
  const __amdgpu_buffer_rsrc_t rl = make_rsrc(lse, (uint32_t)((size_t)gridDim.z * H * S * 4));
  const uint32_t qbase = (uint32_t)(((size_t)b * S * ld + hh * HD) * 2);
  const uint32_t lbase = (uint32_t)(((size_t)b * H + hh) * S * 4);
  auto load = [&](int t, int s) {
    tile_load<HD, NW>(rq, qbase, (uint32_t)ld, t * KT, smem + s * TE);
    const uint32_t lo = lbase + (uint32_t)(t * KT + lane) * 4u;
    if (wid == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_ptr_t*)(fsm + s * KT), 4, lo, 0, 0, 0);
  };
  float csum = 0.f;
  auto unit = [&](int s, int u, int q0, auto rag) {
    const bf16_t* Qs = smem + s * TE;
    f32x16 sv;
    zero16(sv);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) sv = mfma(row_frag<HD>(Qs, u * 32, ks), kf[ks], sv);
    const float* ls = fsm + s * KT + u * 32;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int ql = srow(r, h32);
      float p = ex2(fmaf(sv[r], sl2, -ls[ql]));
      if constexpr (decltype(rag)::value) {
        if (q0 + ql >= S) p = 0.f;
      }
      csum += p;
    }
  };

  load(0, 0);
  if (nt > 1) load(1, 1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  auto tile = [&](int t, auto stg) {
    constexpr int s0 = decltype(stg)::value, s2 = (s0 + 2) % NSTG;
    const bool rag = ragged && t + 1 == nt;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      if (rag) unit(s0, u, t * KT + u * 32, std::true_type{});
      else unit(s0, u, t * KT + u * 32, std::false_type{});
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();   // tile t+1 resident; tile t's stage no longer read
    if (t + 2 < nt) load(t + 2, s2);
  };
  int t = 0;
  for (; t + NSTG <= nt; t += NSTG) {
    tile(t, IC<0>{});
    tile(t + 1, IC<1>{});
    tile(t + 2, IC<2>{});
  }
  if (t < nt) tile(t, IC<0>{});
  if (t + 1 < nt) tile(t + 1, IC<1>{});
  __builtin_amdgcn_s_waitcnt(0);

  csum += __shfl_xor(csum, 32, 64);
  if (h32 == 0 && mykey < S) colsum[((size_t)b * H + hh) * S + mykey] = csum;
}

template <typename Ta, int HDT>
__global__ __launch_bounds__(64) void attn_colsum_simple(const Ta* __restrict__ qkv, const float* __restrict__ lse,
                                                         float* __restrict__ colsum, int S, int H, int D,
                                                         float sl2) {
  const int b = blockIdx.z, hh = blockIdx.y;
  const int k = blockIdx.x * 64 + threadIdx.x;
  if (k >= S) return;
  const size_t ld = 3 * (size_t)D;
  const Ta* base = qkv + (size_t)b * S * ld;
  float kv[HDT];
#pragma unroll
  for (int d = 0; d < HDT; ++d) kv[d] = to_f32<Ta>(base[(size_t)k * ld + D + hh * HDT + d]);
  float acc = 0.f;
  for (int q = 0; q < S; ++q) {
    const Ta* qr = base + (size_t)q * ld + hh * HDT;
    float s = 0.f;
#pragma unroll
    for (int d = 0; d < HDT; ++d) s = fmaf(to_f32<Ta>(qr[d]), kv[d], s);
    acc += exp2f(s * sl2 - lse[((size_t)b * H + hh) * S + q]);
  }
  colsum[((size_t)b * H + hh) * S + k] = acc;
}

// ------------------------------------------------------------------------------ launchers

static inline float attn_sl2(int hd) { return 1.4426950408889634f / sqrtf((float)hd); }

bool attn_uses_mfma(int dtype, int hd) { return dtype == kBF16 && (hd == 64 || hd == 128); }

template <typename Ta>
static hipError_t fwd_simple(const Ta* qkv, Ta* O, float* lse, int B, int S, int H, int D, int hd, hipStream_t st) {
  dim3 g((S + 63) / 64, H, B);
  const float sl2 = attn_sl2(hd);
  if (hd == 32) SR_LAUNCH((attn_fwd_simple<Ta, 32>), g, dim3(64), 0, st, qkv, O, lse, S, H, D, sl2);
  else if (hd == 64) SR_LAUNCH((attn_fwd_simple<Ta, 64>), g, dim3(64), 0, st, qkv, O, lse, S, H, D, sl2);
  else SR_LAUNCH((attn_fwd_simple<Ta, 128>), g, dim3(64), 0, st, qkv, O, lse, S, H, D, sl2);
  return hipGetLastError();
}

template <typename Ta>
static hipError_t bwd_simple(const Ta* qkv, const Ta* dO, const float* lse, const float* delta, Ta* dqkv, int B,
                             int S, int H, int D, int hd, hipStream_t st) {
  dim3 g((S + 63) / 64, H, B);
  const float sl2 = attn_sl2(hd), sc = 1.0f / sqrtf((float)hd);
#define SR_ABS(HDV)                                                                                              \
  SR_LAUNCH((attn_bwd_dq_simple<Ta, HDV>), g, dim3(64), 0, st, qkv, dO, lse, delta, dqkv, S, H, D, sl2, sc); \
  SR_LAUNCH((attn_bwd_dkv_simple<Ta, HDV>), g, dim3(64), 0, st, qkv, dO, lse, delta, dqkv, S, H, D, sl2, sc)
  if (hd == 32) { SR_ABS(32); } else if (hd == 64) { SR_ABS(64); } else { SR_ABS(128); }
#undef SR_ABS
  return hipGetLastError();
}

#define SR_TRY_HIP(x)                 \
  do {                                \
    hipError_t e_ = (x);              \
    if (e_ != hipSuccess) return e_;  \
  } while (0)

// The MFMA kernels on Sq query rows and Skv key/value rows (self-attention: both S, q, k and v
// in one token-major qkv buffer; asymmetric attention: separate buffers).
template <int HD>
static hipError_t fwd_mfma_hd(const bf16_t* q, int ldq, const bf16_t* kv, int ldkv, uint32_t kv_elems, bf16_t* O,
                              float* lse, int B, int Sq, int Skv, int H, int D, hipStream_t st) {
  constexpr int kw = attn_waves<HD>();
  dim3 g((Sq + 32 * kw - 1) / (32 * kw), H, B);
  if constexpr (HD == 128)
    SR_LAUNCH(attn_fwd_h128, g, dim3(64 * kw), 0, st, q, ldq, kv, ldkv, kv_elems, O, lse, Sq, Skv, H, D,
                       attn_sl2(HD));
  else
    SR_LAUNCH((attn_fwd_mfma<HD, kw>), g, dim3(64 * kw), 0, st, q, ldq, kv, ldkv, kv_elems, O, lse, Sq, Skv,
                       H, D, attn_sl2(HD));
  return hipGetLastError();
}

hipError_t launch_attn_fwd_mfma(const bf16_t* q, int ldq, const bf16_t* kv, int ldkv, uint32_t kv_elems, bf16_t* O,
                                float* lse, int B, int Sq, int Skv, int H, int D, hipStream_t st) {
  if (D / H == 128) return fwd_mfma_hd<128>(q, ldq, kv, ldkv, kv_elems, O, lse, B, Sq, Skv, H, D, st);
  return fwd_mfma_hd<64>(q, ldq, kv, ldkv, kv_elems, O, lse, B, Sq, Skv, H, D, st);
}

template <int HD>
static hipError_t dkv_mfma_hd(const bf16_t* q, int ldq, uint32_t q_elems, const bf16_t* kv, int ldkv,
                              const bf16_t* dO, const float* lse, const float* delta, bf16_t* dk_out, int ldo, int B,
                              int Sq, int Skv, int H, int D, hipStream_t st) {
  constexpr int kw = attn_waves<HD>();
  dim3 g((Skv + 32 * kw - 1) / (32 * kw), H, B);
  if constexpr (HD == 128)
    SR_LAUNCH(attn_bwd_dkv_h128, g, dim3(64 * kw), 0, st, q, ldq, q_elems, kv, ldkv, dO, lse, delta, dk_out,
                       ldo, Sq, Skv, H, D, attn_sl2(HD), 1.0f / sqrtf((float)HD));
  else
    SR_LAUNCH((attn_bwd_dkv_mfma<HD, kw>), g, dim3(64 * kw), 0, st, q, ldq, q_elems, kv, ldkv, dO, lse,
                       delta, dk_out, ldo, Sq, Skv, H, D, attn_sl2(HD), 1.0f / sqrtf((float)HD));
  return hipGetLastError();
}

hipError_t launch_attn_dkv_mfma(const bf16_t* q, int ldq, uint32_t q_elems, const bf16_t* kv, int ldkv,
                                const bf16_t* dO, const float* lse, const float* delta, bf16_t* dk_out, int ldo, int B,
                                int Sq, int Skv, int H, int D, hipStream_t st) {
  if (D / H == 128)
    return dkv_mfma_hd<128>(q, ldq, q_elems, kv, ldkv, dO, lse, delta, dk_out, ldo, B, Sq, Skv, H, D, st);
  return dkv_mfma_hd<64>(q, ldq, q_elems, kv, ldkv, dO, lse, delta, dk_out, ldo, B, Sq, Skv, H, D, st);
}

template <int HD>
static hipError_t dq_mfma_hd(const bf16_t* q, int ldq, const bf16_t* kv, int ldkv, uint32_t kv_elems,
                             const bf16_t* dO, const float* lse, const float* delta, bf16_t* dq_out, int ldo, int B,
                             int Sq, int Skv, int H, int D, hipStream_t st) {
  constexpr int kw = attn_waves<HD>();
  dim3 g((Sq + 32 * kw - 1) / (32 * kw), H, B);
  if constexpr (HD == 128)
    SR_LAUNCH(attn_bwd_dq_h128, g, dim3(64 * kw), 0, st, q, ldq, kv, ldkv, kv_elems, dO, lse, delta, dq_out,
                       ldo, Sq, Skv, H, D, attn_sl2(HD), 1.0f / sqrtf((float)HD));
  else
    SR_LAUNCH((attn_bwd_dq_mfma<HD, kw>), g, dim3(64 * kw), 0, st, q, ldq, kv, ldkv, kv_elems, dO, lse,
                       delta, dq_out, ldo, Sq, Skv, H, D, attn_sl2(HD), 1.0f / sqrtf((float)HD));
  return hipGetLastError();
}

hipError_t launch_attn_dq_mfma(const bf16_t* q, int ldq, const bf16_t* kv, int ldkv, uint32_t kv_elems,
                               const bf16_t* dO, const float* lse, const float* delta, bf16_t* dq_out, int ldo, int B,
                               int Sq, int Skv, int H, int D, hipStream_t st) {
  if (D / H == 128)
    return dq_mfma_hd<128>(q, ldq, kv, ldkv, kv_elems, dO, lse, delta, dq_out, ldo, B, Sq, Skv, H, D, st);
  return dq_mfma_hd<64>(q, ldq, kv, ldkv, kv_elems, dO, lse, delta, dq_out, ldo, B, Sq, Skv, H, D, st);
}

hipError_t launch_attn_fwd(int dtype, const void* qkv, void* O, float* lse, int B, int S, int H, int D,
                           hipStream_t st) {
  const int hd = D / H;
  if (attn_uses_mfma(dtype, hd)) {
    const bf16_t* q = (const bf16_t*)qkv;
    return launch_attn_fwd_mfma(q, 3 * D, q + D, 3 * D, (uint32_t)((size_t)B * S * 3 * D - D), (bf16_t*)O, lse, B,
                                S, S, H, D, st);
  }
  if (dtype == kBF16) return fwd_simple((const bf16_t*)qkv, (bf16_t*)O, lse, B, S, H, D, hd, st);
  return fwd_simple((const float*)qkv, (float*)O, lse, B, S, H, D, hd, st);
}

hipError_t launch_attn_bwd(int dtype, const void* qkv, const void* dO, const float* lse, const float* delta,
                           void* dqkv, int B, int S, int H, int D, hipStream_t st) {
  const int hd = D / H;
  if (attn_uses_mfma(dtype, hd)) {
    const float sl2 = attn_sl2(hd), sc = 1.0f / sqrtf((float)hd);
    const double units = 2.0 * B * (double)S * S * D;   // one S x S x hd product over all heads
    const bf16_t* q = (const bf16_t*)qkv;
    const uint32_t all = (uint32_t)((size_t)B * S * 3 * D);
    {
      // algorithmic: dP, dV, dK (the recomputed scores are not counted)
      ProfScope ps("attn_bwd_dkv", 3 * units, (double)B * S * D * 2 * 6, st);
      SR_TRY_HIP(launch_attn_dkv_mfma(q, 3 * D, all, q + D, 3 * D, (const bf16_t*)dO, lse, delta, (bf16_t*)dqkv + D,
                                      3 * D, B, S, S, H, D, st));
    }
    {
      ProfScope ps("attn_bwd_dq", units, (double)B * S * D * 2 * 5, st);
      SR_TRY_HIP(launch_attn_dq_mfma(q, 3 * D, q + D, 3 * D, all - D, (const bf16_t*)dO, lse, delta, (bf16_t*)dqkv,
                                     3 * D, B, S, S, H, D, st));
    }
    (void)sl2; (void)sc;
    return hipSuccess;
  }
  ProfScope ps("attn_bwd_generic", 8.0 * B * (double)S * S * D, 0, st);
  if (dtype == kBF16)
    return bwd_simple((const bf16_t*)qkv, (const bf16_t*)dO, lse, delta, (bf16_t*)dqkv, B, S, H, D, hd, st);
  return bwd_simple((const float*)qkv, (const float*)dO, lse, delta, (float*)dqkv, B, S, H, D, hd, st);
}

template <typename Ta>
static hipError_t colsum_simple(const Ta* qkv, const float* lse, float* colsum, int B, int S, int H, int D, int hd,
                                hipStream_t st) {
  dim3 g((S + 63) / 64, H, B);
  const float sl2 = attn_sl2(hd);
  if (hd == 32) SR_LAUNCH((attn_colsum_simple<Ta, 32>), g, dim3(64), 0, st, qkv, lse, colsum, S, H, D, sl2);
  else if (hd == 64) SR_LAUNCH((attn_colsum_simple<Ta, 64>), g, dim3(64), 0, st, qkv, lse, colsum, S, H, D, sl2);
  else SR_LAUNCH((attn_colsum_simple<Ta, 128>), g, dim3(64), 0, st, qkv, lse, colsum, S, H, D, sl2);
  return hipGetLastError();
}

hipError_t launch_attn_colsum(int dtype, const void* qkv, const float* lse, float* colsum, int B, int S, int H, int D,
                              hipStream_t st) {
  const int hd = D / H;
  if (dtype == kBF16 && hd == 64) {   // MFMA column sums at head dim 64; other head dims generic
    constexpr int kw = attn_waves<64>();   // the dK/dV kernel's score half: the same shape
    dim3 g((S + 32 * kw - 1) / (32 * kw), H, B);
    SR_LAUNCH(attn_colsum_mfma<kw>, g, dim3(64 * kw), 0, st, (const bf16_t*)qkv, lse, colsum, S, H, D,
                       attn_sl2(hd));
    return hipGetLastError();
  }
  if (dtype == kBF16) return colsum_simple((const bf16_t*)qkv, lse, colsum, B, S, H, D, hd, st);
  return colsum_simple((const float*)qkv, lse, colsum, B, S, H, D, hd, st);
}

}  // namespace sr
