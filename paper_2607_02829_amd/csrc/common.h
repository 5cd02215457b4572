// Device-side helpers shared by the gfx950 kernels of libsr.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sr {
// Completion events bound to kernels at launch.  Every kernel of the library is launched through
// SR_LAUNCH.  While the calling thread's hook holds a stop event, each launch carries it (and the
// start event, on the first launch only) with hipExtLaunchKernelGGL, so the events mark that
// kernel's own start and end.  A separate event record between two kernels of one stream is a
// marker packet that leaves the stream idle for several microseconds; a bound event costs about
// a third of that.  Used for the timing of profiled launch groups and for the forks of the
// backward's second stream (the side stream then waits on the event of the last kernel it needs).
struct LaunchHook {
  hipEvent_t start = nullptr;          // bound to the next launch only
  hipEvent_t stop = nullptr;           // bound to every launch while set
  hipStream_t last_stream = nullptr;   // stream and stop event of the most recent launch
  hipEvent_t last_stop = nullptr;
  unsigned long long launches = 0;     // launches through SR_LAUNCH on this thread
};
LaunchHook& launch_hook();   // per thread

template <typename F, typename... A>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t st, A... args) {
  LaunchHook& h = launch_hook();
  if (h.stop) {
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, h.start, h.stop, 0, args...);
    h.start = nullptr;
  } else {
    hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
  }
  h.last_stream = st;
  h.last_stop = h.stop;
  ++h.launches;
}
}  // namespace sr
#define SR_LAUNCH(kernel, ...) ::sr::launch_kernel((kernel), __VA_ARGS__)

typedef uint16_t bf16_t;   // bfloat16 bit pattern in memory

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;
typedef __attribute__((__vector_size__(2 * sizeof(int)))) int i32x2;

#define SR_DEV __device__ __forceinline__

// ---------------------------------------------------------------- conversions
SR_DEV float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// fp32 -> bf16 with the hardware conversion (v_cvt_pk_bf16_f32): round to nearest even,
// denormals kept, NaN stays NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Packed pair (lo in bits 0..15).
SR_DEV uint32_t f2bf2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
SR_DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

template <typename T> SR_DEV float to_f32(T v);
template <> SR_DEV float to_f32<float>(float v) { return v; }
template <> SR_DEV float to_f32<bf16_t>(bf16_t v) { return bf2f(v); }

template <typename T> SR_DEV T from_f32(float v);
template <> SR_DEV float from_f32<float>(float v) { return v; }
template <> SR_DEV bf16_t from_f32<bf16_t>(float v) { return f2bf(v); }

// The wave's index in its workgroup as a wave-uniform (scalar) value, so that addresses derived
// from it (LDS blocks, M0) stay in scalar registers.
SR_DEV int wave_index() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// ---------------------------------------------------------------- wave reductions
// Every lane ends with the same (bitwise) result: DPP exchanges within 16-lane rows
// (pairs, quads, half-row mirror, row mirror), then v_permlane16_swap / v_permlane32_swap
// between rows; no LDS round trips.
template <int CTRL>
SR_DEV float dppf(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
SR_DEV float wave_sum(float v) {
  v += dppf<0xB1>(v);    // quad_perm(1,0,3,2)
  v += dppf<0x4E>(v);    // quad_perm(2,3,0,1)
  v += dppf<0x141>(v);   // row_half_mirror
  v += dppf<0x140>(v);   // row_mirror
  {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return v;
}
// v combined with the value of the lane 32 apart (the two halves of a wave).
SR_DEV float half_pair_sum(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
SR_DEV float half_pair_max(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
SR_DEV float wave_max(float v) {
  v = fmaxf(v, dppf<0xB1>(v));
  v = fmaxf(v, dppf<0x4E>(v));
  v = fmaxf(v, dppf<0x141>(v));
  v = fmaxf(v, dppf<0x140>(v));
  {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  return v;
}

// ---------------------------------------------------------------- buffer resources
// Raw buffer loads return zero for any byte offset at or beyond num_records, which
// gives zero-filled ragged tails without per-element predicates.
SR_DEV __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t nbytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)nbytes, 0x00020000);
}
SR_DEV i32x4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
SR_DEV i32x2 buf_load8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0);
}

// LDS address space, for the loads that write LDS directly (buffer_load ... lds) and the
// transposing LDS reads.
typedef __attribute__((address_space(3))) void lds_ptr_t;

// Transposing LDS read (ds_read_b64_tr_b16): the 16 lanes of each group address four rows
// of 16 bf16 (lane s: row s / 4, elements 4 (s % 4) .. + 3) and lane s receives element s of
// each of the four rows.
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
SR_DEV v4s ds_tr(const bf16_t* p) { return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)p); }

template <int V>
struct IC {
  static constexpr int value = V;
};

template <int N, typename F>
SR_DEV void static_for(F&& f) {
  if constexpr (N > 0) {
    static_for<N - 1>(f);
    f(IC<N - 1>{});
  }
}

// s_waitcnt with vmcnt <= N (buffer loads, including those that write LDS directly) and
// lgkmcnt = 0 (LDS reads), expcnt untouched.
template <int N>
SR_DEV void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | ((N >> 4) << 14));
}

// ---------------------------------------------------------------- explicit LDS reads
// Fragment reads written as inline asm: the compiler then does not treat them as LDS
// accesses that might alias a global->LDS fill still in flight (it would wait for every
// outstanding fill before each read).  Their completion is not tracked by the compiler
// either: callers wait with lgkm_wait<N>() and pin the destination registers behind it.
SR_DEV uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}
template <int OFF>
SR_DEV i32x4 lds_read16(uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x4 v;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}
template <int OFF>
SR_DEV i32x2 lds_read_tr8(uint32_t a) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x2 v;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(v) : "v"(a), "i"(OFF));
  return v;
}
// Explicit LDS reads at a compile-time byte offset (the 16-bit instruction offset field takes
// what fits, the rest is added to the address).
template <int OFF>
SR_DEV i32x4 rd16(uint32_t a) {
  constexpr int HI = OFF & ~0xFFFF;
  return lds_read16<OFF - HI>(a + HI);
}
template <int OFF>
SR_DEV i32x2 rdtr(uint32_t a) {
  constexpr int HI = OFF & ~0xFFFF;
  return lds_read_tr8<OFF - HI>(a + HI);
}

template <int N>
SR_DEV void lgkm_wait() {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N));
}
template <typename V>
SR_DEV void pin(V& v) {
  asm volatile("" : "+v"(v));
}

// Raw fragment as the explicit reads deliver it: one 16-byte read (k-major) or two 8-byte
// transposing reads (r-major).  The registers are written asynchronously, so nothing may touch
// them before lgkm_wait: settle() pins each destination behind the wait and only then joins the
// halves into the MFMA operand.
template <bool KMAJ>
struct RawFrag;
template <>
struct RawFrag<true> {
  i32x4 v;
  SR_DEV bf16x8 settle() {
    pin(v);
    return __builtin_bit_cast(bf16x8, v);
  }
};
template <>
struct RawFrag<false> {
  i32x2 lo, hi;
  SR_DEV bf16x8 settle() {
    pin(lo);
    pin(hi);
    i32x4 w;
    w[0] = lo[0]; w[1] = lo[1]; w[2] = hi[0]; w[3] = hi[1];
    return __builtin_bit_cast(bf16x8, w);
  }
};

// Workgroup barrier as inline asm.  The compiler makes every global->LDS fill still in flight
// complete before a barrier it can see (s_waitcnt vmcnt(0)), which would drain a multi-stage
// fill pipeline at every tile; callers of this one wait explicitly for exactly the fills (and
// LDS reads) that must be complete.
SR_DEV void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }
