// Launch sequences of the middle-block stack (Eq. sparse_forward; block of
// Sec. 3.3) and of its vector-Jacobian product.
//
// Forward, per block (pre-LN; adaLN replaces the LN affine by the per-sample
// modulation and gates the two residual branches):
//   u1 = LN1(h)                      rowops  ln_fwd (routed calls: the first block's reads the
//                                                    rows x[idx] itself, ln_fwd_gather)
//   qkv = u1 W_qkv^T + b_qkv         gemm    EPI_BIAS_ACT
//   O, lse = attention(qkv)          attention fwd
//   h1 = h + O W_o^T + b_o           gemm    EPI_RESID
//   u2 = LN2(h1)                     rowops  ln_fwd
//   z, g = GELU(u2 W1^T + b1)        gemm    EPI_GELU
//   h' = h1 + g W2^T + b2            gemm    EPI_RESID (fp32 residual stream; last block
//                                                      rounds to the storage type once)
// Backward runs the same steps in reverse (dW by split-K GEMMs over tokens with a
// deterministic partial-sum reduction; bias / LN / modulation gradients by
// chunked column sums).  The weight-gradient GEMMs are off the critical path: they run
// on a second stream of the device, forked from the caller's stream after their inputs
// are written and joined before those inputs are overwritten (and at the end), so they
// fill the tails of the dX GEMMs, LayerNorms and attention kernels.
#include "stack.h"

#include <cmath>
#include <mutex>
#include <vector>

#include "common.h"
#include "profile.h"

namespace sr {

namespace {

struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(char* b) : base(b) {}
  template <typename P>
  P* take(size_t bytes) {
    off = (off + 255) & ~(size_t)255;
    P* p = base ? reinterpret_cast<P*>(base + off) : nullptr;
    off += bytes;
    return p;
  }
};

#define SR_TRY(x)                           \
  do {                                      \
    hipError_t _e = (x);                    \
    if (_e != hipSuccess) return _e;        \
  } while (0)

// Algorithmic work of a launch group, for the optional event timing.
double gemm_flops(int M, int N, int K) { return 2.0 * M * N * K; }
double gemm_bytes(const Dims& d, int M, int N, int K, int out_elt) {
  return ((double)M * K + (double)N * K) * d.elt + (double)M * N * out_elt;
}

GemmDesc desc(const Dims& d, const void* A, bool ak, long long lda, size_t abytes, const void* B, bool bk,
              long long ldb, size_t bbytes, int M, int N, int K) {
  GemmDesc g;
  g.A = A; g.B = B; g.M = M; g.N = N; g.K = K;
  g.lda = lda; g.ldb = ldb; g.a_bytes = abytes; g.b_bytes = bbytes;
  g.a_kmajor = ak; g.b_kmajor = bk;
  g.use_mfma = d.dtype == kBF16;
  g.dtype = d.dtype;
  g.a_type = d.dtype; g.b_type = d.dtype;
  return g;
}

}  // namespace

// Per block: what the backward reads.  The LayerNorm outputs u1, u2 and GELU(z) are forward
// temporaries shared by all blocks (the backward recomputes them from the fp32 residual stream
// and the saved statistics, and from z, bit for bit), 12 of the 36.9 KB per token and block at
// D = 1024.
size_t layout_saved(const Dims& d, char* base, BlockSaved* out) {
  Carver c(base);
  const size_t M = d.M, D = d.D, F = d.F, e = d.elt;
  for (int i = 0; i < d.nb; ++i) {
    BlockSaved s{};
    s.hin = c.take<float>(M * D * 4);
    s.mean1 = c.take<float>(M * 4);
    s.rstd1 = c.take<float>(M * 4);
    s.qkv = c.take<void>(M * 3 * D * e);
    s.O = c.take<void>(M * D * e);
    s.lse = c.take<float>((size_t)d.B * d.H * d.S * 4);
    s.h1 = c.take<float>(M * D * 4);
    s.mean2 = c.take<float>(M * 4);
    s.rstd2 = c.take<float>(M * 4);
    s.z = c.take<void>(M * F * e);
    if (d.kind == SR_BLOCK_ADALN) {
      s.mod = c.take<float>((size_t)d.B * 6 * D * 4);
      s.a_out = c.take<void>(M * D * e);
      s.m_out = c.take<void>(M * D * e);
    }
    if (out) out[i] = s;
  }
  void* u_tmp = c.take<void>(M * D * e);
  void* gz_tmp = c.take<void>(M * F * e);
  if (out)
    for (int i = 0; i < d.nb; ++i) { out[i].u1 = out[i].u2 = u_tmp; out[i].gz = gz_tmp; }
  return c.off;
}

// weight-gradient kinds: rows and columns of dW as {0: 3D, 1: D, 2: F} and {1: D, 2: F}
enum { kWgQkv = 0, kWgO = 1, kWgFc1 = 2, kWgFc2 = 3 };
static const int kWeightGradShapes[4][2] = {{0, 1}, {1, 1}, {2, 1}, {1, 2}};

size_t layout_scratch(const Dims& d, char* base, Scratch* out) {
  Carver c(base);
  const size_t M = d.M, D = d.D, F = d.F, e = d.elt;
  Scratch s{};
  s.g_res = c.take<float>(M * D * 4);
  s.g_res2 = c.take<float>(M * D * 4);
  s.du = c.take<float>(M * D * 4);
  s.delta = c.take<float>((size_t)d.B * d.H * d.S * 4);
  for (int k = 0; k < 4; ++k) {
    const int* sh = kWeightGradShapes[k];
    const int rows = sh[0] == 0 ? 3 * d.D : sh[0] == 1 ? d.D : d.F, cols = sh[1] == 1 ? d.D : d.F;
    size_t pf = 0, df = 0;
    if (d.dtype == kBF16) weight_grad_scratch(rows, cols, d.M, &pf, &df);
    s.wpart[k] = c.take<float>((pf + (size_t)rows * cols) * 4);   // split partials, then an unwanted dW
    s.dbpart[k] = c.take<float>(std::max<size_t>(df, 1) * 4);
  }
  const size_t wmax = std::max<size_t>(std::max<size_t>(3 * D, F), 6 * D);
  s.part = c.take<float>((size_t)d.B * colsum_chunks(d.S) * wmax * 4);
  // LayerNorm parameter-gradient partials of LN2 and LN1, two of each by block parity (pre-LN:
  // their reductions run on the side stream, one or two blocks after the partials are written)
  for (int k = 0; k < 2; ++k)
    for (int q = 0; q < 2; ++q) s.lnpart[k][q] = c.take<float>((size_t)d.B * ln_bwd_chunks(d.S) * 2 * D * 4);
  s.dmod = c.take<float>((size_t)d.B * 6 * D * 4);
  s.gvpart = d.kind == SR_BLOCK_ADALN ? c.take<float>(gemv_cols_scratch(d.B, 6 * d.D, d.D) * 4) : nullptr;
  // two of each buffer a weight-gradient GEMM reads on the side stream, so the main stream
  // rarely waits for it before writing the next one
  for (int k = 0; k < 2; ++k) s.g_act[k] = c.take<void>(M * D * e);
  for (int k = 0; k < 2; ++k) s.dz[k] = c.take<void>(M * F * e);
  s.dO = c.take<void>(M * D * e);
  for (int k = 0; k < 2; ++k) s.dqkv[k] = c.take<void>(M * 3 * D * e);
  // recomputed operands of the weight-gradient GEMMs (written and read on the second stream)
  s.u_rc = c.take<void>(M * D * e);
  s.gz_rc = c.take<void>(M * F * e);
  if (out) *out = s;
  return c.off;
}

// ============================================================================ forward

hipError_t stack_fwd(const Dims& d, const sr_block_params* p, const void* cond, const void* h_in, void* h_out,
                     char* saved, hipStream_t st, const Route* rt) {
  BlockSaved* sv = new BlockSaved[d.nb];
  layout_saved(d, saved, sv);
  const int M = d.M, D = d.D, F = d.F, S = d.S;
  const size_t e = d.elt;
  const bool ada = d.kind == SR_BLOCK_ADALN;
  hipError_t err = hipSuccess;
  auto run = [&]() -> hipError_t {
    if (!rt) {   // the fp32 residual stream from h_in (routed calls gather it in the first LayerNorm)
      ProfScope ps("convert", 0, (double)M * D * (e + 4), st);
      SR_TRY(launch_convert(d.dtype, h_in, kF32, sv[0].hin, (size_t)M * D, nullptr, 0, S, D, nullptr, st));
    }
    for (int i = 0; i < d.nb; ++i) {
      const BlockSaved& s = sv[i];
      const sr_block_params& w = p[i];
      if (ada) {   // mod_b = c_b W_ada^T + b_ada
        ProfScope ps("mod", gemm_flops(d.B, 6 * D, D), gemm_bytes(d, d.B, 6 * D, D, 4), st);
        SR_TRY(launch_gemv_rows(d.dtype, cond, D, w.w_ada, w.b_ada, d.B, 6 * D, D, s.mod, 6 * D, st));
      }
      if (rt && i == 0) {   // x[idx] rows -> fp32 residual copy and LN1, one pass
        ProfScope ps("ln_fwd_gather", 0, (double)M * D * (2 * e + 4) + 4.0 * M, st);
        SR_TRY(launch_ln_fwd_gather(d.dtype, rt->x, rt->idx, d.L, rt->shared, s.hin, w.ln1_w, w.ln1_b,
                                    ada ? s.mod : nullptr, 0, M, S, D, d.eps, s.u1, s.mean1, s.rstd1, st));
      } else {
        ProfScope ps("ln_fwd", 0, (double)M * D * (4 + e), st);
        SR_TRY(launch_ln_fwd(d.dtype, s.hin, w.ln1_w, w.ln1_b, ada ? s.mod : nullptr, 0, M, S, D, d.eps, s.u1,
                             s.mean1, s.rstd1, st));
      }
      {
        GemmDesc g = desc(d, s.u1, true, D, (size_t)M * D * e, w.w_qkv, true, D, (size_t)3 * D * D * e, M, 3 * D, D);
        EpiArgs ep; ep.out_act = s.qkv; ep.bias = w.b_qkv; ep.ldo = 3 * D;
        ProfScope ps("gemm_qkv", gemm_flops(M, 3 * D, D), gemm_bytes(d, M, 3 * D, D, (int)e), st);
        SR_TRY(launch_gemm(g, EPI_BIAS_ACT, ep, st));
      }
      {
        ProfScope ps("attn_fwd", 4.0 * d.B * (double)S * S * D, (double)M * D * e * 4, st);
        SR_TRY(launch_attn_fwd(d.dtype, s.qkv, s.O, s.lse, d.B, S, d.H, D, st));
      }
      {
        GemmDesc g = desc(d, s.O, true, D, (size_t)M * D * e, w.w_o, true, D, (size_t)D * D * e, M, D, D);
        EpiArgs ep; ep.bias = w.b_o; ep.resid = s.hin; ep.out_f32 = s.h1; ep.ldo = D; ep.S = S;
        if (ada) { ep.gate = s.mod + 2 * D; ep.gate_stride = 6 * D; ep.a_save = s.a_out; }
        ProfScope ps("gemm_o", gemm_flops(M, D, D), gemm_bytes(d, M, D, D, 8), st);
        SR_TRY(launch_gemm(g, EPI_RESID, ep, st));
      }
      {
        ProfScope ps("ln_fwd", 0, (double)M * D * (4 + e), st);
        SR_TRY(launch_ln_fwd(d.dtype, s.h1, w.ln2_w, w.ln2_b, ada ? s.mod : nullptr, 3 * D, M, S, D, d.eps, s.u2,
                             s.mean2, s.rstd2, st));
      }
      {
        GemmDesc g = desc(d, s.u2, true, D, (size_t)M * D * e, w.w_fc1, true, D, (size_t)F * D * e, M, F, D);
        EpiArgs ep; ep.bias = w.b_fc1; ep.out_act = s.z; ep.out_act2 = s.gz; ep.ldo = F;
        ProfScope ps("gemm_fc1", gemm_flops(M, F, D), gemm_bytes(d, M, F, D, 2 * (int)e), st);
        SR_TRY(launch_gemm(g, EPI_GELU, ep, st));
      }
      {
        GemmDesc g = desc(d, s.gz, true, F, (size_t)M * F * e, w.w_fc2, true, F, (size_t)D * F * e, M, D, F);
        EpiArgs ep; ep.bias = w.b_fc2; ep.resid = s.h1; ep.ldo = D; ep.S = S;
        if (i + 1 < d.nb) {
          ep.out_f32 = sv[i + 1].hin;
        } else if (rt) {   // x[I] = rnd(x0 + (rnd(h) - x0)) in the epilogue
          ep.sc_x = rt->x; ep.sc_idx = rt->idx; ep.sc_L = d.L; ep.sc_shared = rt->shared;
        } else {
          ep.out_st = h_out;
        }
        if (ada) { ep.gate = s.mod + 5 * D; ep.gate_stride = 6 * D; ep.a_save = s.m_out; }
        ProfScope ps("gemm_fc2", gemm_flops(M, D, F), gemm_bytes(d, M, D, F, 8), st);
        SR_TRY(launch_gemm(g, EPI_RESID, ep, st));
      }
    }
    return hipSuccess;
  };
  err = run();
  delete[] sv;
  return err;
}

// ============================================================================ backward

namespace {

// dW[N x K] = sum_m dY[m, n] X[m, k] and db[n] = sum_m dY[m, n], both operands token-major
// ([M, N] and [M, K]); the GEMM layer picks the tile shape and any split over tokens.
// The reduction it needs (split planes, bias partial rows) is left in *job, for one launch per
// block (launch_reduce_jobs).
hipError_t weight_grad(const char* name, const Dims& d, const void* dY, int N, const void* X, int K, float* out,
                       float* db, const Scratch& sc, int kind, ReduceJob* job, hipStream_t st) {
  *job = ReduceJob{};
  if (!out && !db) return hipSuccess;
  const size_t e = d.elt;
  GemmDesc g = desc(d, dY, false, N, (size_t)d.M * N * e, X, false, K, (size_t)d.M * K * e, N, K, d.M);
  size_t pf = 0, df = 0;
  if (g.use_mfma) weight_grad_scratch(N, K, d.M, &pf, &df);
  float* dw = out ? out : sc.wpart[kind] + pf;   // the kernel always produces dW; park an unwanted one
  ProfScope ps(name, gemm_flops(N, K, d.M), gemm_bytes(d, N, K, d.M, 4), st);
  return launch_weight_grad(g, dw, db, sc.wpart[kind], sc.dbpart[kind], st, job);
}

// dmod[b, off + c] = sum_s X[b,s,c] * Y[b,s,c]  (adaLN gate gradients)
hipError_t gate_grad(const Dims& d, const float* X, const void* Y, float* dmod, int off, const Scratch& sc,
                     hipStream_t st) {
  ProfScope ps("colsum", 0, (double)d.M * d.D * (4 + d.elt), st);
  SR_TRY(launch_colsum(kF32, X, d.dtype, Y, nullptr, 0, d.B, d.S, d.D, sc.part, st));
  return launch_reduce_cols(sc.part, colsum_chunks(d.S), d.B, 0, d.D, d.D, dmod + off, nullptr, 6 * d.D, st);
}

hipError_t zero_f32(float* p, size_t n, hipStream_t st) {
  return p ? launch_fill_f32(p, n, 0.0f, st) : hipSuccess;
}

}  // namespace

// One extra stream per device for the weight-gradient work (default priority; created on
// first use and kept for the life of the process).
constexpr int kMaxDevices = 64;
hipError_t side_stream(hipStream_t* out) {
  static hipStream_t streams[kMaxDevices] = {};
  static std::mutex mu;
  int dev = 0;
  SR_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (!streams[dev]) SR_TRY(hipStreamCreateWithFlags(&streams[dev], hipStreamNonBlocking));
  *out = streams[dev];
  return hipSuccess;
}

// Events of one backward call: fork (caller stream -> side stream) and, per slot, the
// completion of the last weight-gradient GEMM that read a double-buffered input (side ->
// caller).  An event is re-recorded only after the waits on its previous record have been
// enqueued.  Sets are created once and kept in a per-device pool (creating events per call
// costs tens of microseconds of host time).
hipError_t BwdEvents::create() {
  SR_TRY(hipEventCreateWithFlags(&fork, hipEventDisableTiming));
  for (hipEvent_t& e : done) SR_TRY(hipEventCreateWithFlags(&e, hipEventDisableTiming));
  return hipSuccess;
}
namespace {
std::mutex g_ev_mu;
std::vector<BwdEvents*> g_ev_pool;
}  // namespace
hipError_t take_events(BwdEvents** out) {
  int dev = 0;
  SR_TRY(hipGetDevice(&dev));
  {
    std::lock_guard<std::mutex> lock(g_ev_mu);
    for (size_t i = 0; i < g_ev_pool.size(); ++i)
      if (g_ev_pool[i]->dev == dev) {
        *out = g_ev_pool[i];
        g_ev_pool.erase(g_ev_pool.begin() + (long)i);
        return hipSuccess;
      }
  }
  BwdEvents* e = new BwdEvents;
  e->dev = dev;
  const hipError_t r = e->create();
  if (r != hipSuccess) {
    delete e;   // the events created so far are leaked: an event-creation failure is fatal anyway
    return r;
  }
  *out = e;
  return hipSuccess;
}
void give_events(BwdEvents* e) {
  if (!e) return;
  std::lock_guard<std::mutex> lock(g_ev_mu);
  g_ev_pool.push_back(e);
}

hipError_t stack_bwd(const Dims& d, const sr_block_params* p, const void* cond, const char* saved,
                     const void* dh_out, void* dh_in, const sr_block_grads* gr, float* dcond, char* scratch,
                     hipStream_t st, const Route* rt) {
  BlockSaved* sv = new BlockSaved[d.nb];
  layout_saved(d, const_cast<char*>(saved), sv);
  Scratch sc;
  layout_scratch(d, scratch, &sc);
  const int M = d.M, D = d.D, F = d.F, S = d.S;
  const size_t e = d.elt;
  const bool ada = d.kind == SR_BLOCK_ADALN;
  const int nln = ln_bwd_chunks(S);

  hipStream_t side = nullptr;
  BwdEvents* ev = nullptr;
  bool pending[kSlots] = {};   // recorded and not yet waited on
  const bool serial = profiling_all();
  // Fork points: the main-stream kernels right before a fork carry the fork event themselves
  // (bound at launch, see LaunchHook), and the fork waits on the event the last of them carries,
  // provided no kernel was launched in between; otherwise it records the event on st.  Not while
  // st is being captured into a graph (event records there become graph nodes).
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  const bool bind = !serial && hipStreamIsCapturing(st, &capture) == hipSuccess &&
                    capture == hipStreamCaptureStatusNone;
  hipEvent_t fork_ev = nullptr;         // event carried by the last kernel of the last fork point
  unsigned long long fork_at = 0;       // launch count right after it
  auto fork_point = [&](auto&& launch) -> hipError_t {
    if (!bind) return launch();
    LaunchHook& h = launch_hook();
    const hipEvent_t outer = h.stop;
    const unsigned long long n0 = h.launches;
    h.stop = outer ? outer : ev->fork;   // an enclosing binding (a timed group) serves the fork too
    const hipError_t r = launch();
    h.stop = outer;
    fork_ev = r == hipSuccess && h.launches > n0 && h.last_stream == st ? h.last_stop : nullptr;
    fork_at = h.launches;
    return r;
  };
  // side stream: wait for everything issued on st so far, run the weight gradient, signal slot
  auto on_side = [&](int slot, auto&& launch) -> hipError_t {
    if (serial) return launch(st);
    if (fork_ev && launch_hook().launches == fork_at) {
      SR_TRY(hipStreamWaitEvent(side, fork_ev, 0));
    } else {
      SR_TRY(hipEventRecord(ev->fork, st));
      SR_TRY(hipStreamWaitEvent(side, ev->fork, 0));
    }
    fork_ev = nullptr;
    SR_TRY(launch(side));
    SR_TRY(hipEventRecord(ev->done[slot], side));
    pending[slot] = true;
    return hipSuccess;
  };
  // st: wait before overwriting the buffer the slot's weight-gradient GEMM reads
  auto join = [&](int slot) -> hipError_t {
    if (pending[slot]) SR_TRY(hipStreamWaitEvent(st, ev->done[slot], 0));
    pending[slot] = false;
    return hipSuccess;
  };
  // slots: g_act[0] (FC2 stage) and g_act[1] (output-projection stage) are read by dW_fc2 and
  // dW_o; dz[i % 2] by dW_fc1 and dqkv[i % 2] by dW_qkv of block i
  enum { kFc2 = 0, kO = 1, kFc1 = 2, kQkv = 4 };


  // pre-LN: the LayerNorm parameter gradients (column sums of the ln_bwd partials) are outputs
  // only, so their reductions join the block's weight-gradient reductions in the one launch on
  // the side stream after dW_qkv: LN2's of the same block, LN1's of the block before it in
  // backward order (its LN1 backward runs after that launch is forked); the last LN1's at the
  // end.  The partials alternate between two buffers by block parity: the next write of a
  // buffer (two blocks later) follows the join that guards g1 (LN2) or g0 (LN1) of that block,
  // which waits for side-stream work queued after the launch that read it.
  auto ln_job = [&](const float* part, float* dw, float* dbeta) {
    ReduceJob j;
    j.part = part; j.rows = d.B * nln; j.width = 2 * D; j.half = D; j.out = dw; j.dbout = dbeta;
    return j;
  };
  const sr_block_grads* ln1_pending = nullptr;   // block whose LN1 reduction is still to run
  const float* ln1_pending_part = nullptr;

  auto run = [&]() -> hipError_t {
    SR_TRY(side_stream(&side));
    SR_TRY(take_events(&ev));
    // g_res = fp32(dh_out) and, for pre-LN, its activation copy
    if (rt) {   // gather of the gradient fused with its conversion
      ProfScope ps("gather_f32", 0, (double)M * D * (2 * e + 4) + 4.0 * M, st);
      SR_TRY(launch_gather_rows_f32(d.dtype, d.B, d.L, S, D, rt->x, rt->idx, sc.g_res, sc.g_act[0], rt->shared, st));
    } else {
      ProfScope ps("convert", 0, (double)M * D * (2 * e + 4), st);
      SR_TRY(launch_convert(d.dtype, dh_out, d.dtype, sc.g_act[0], (size_t)M * D, nullptr, 0, S, D, sc.g_res, st));
    }
    void* const g0 = sc.g_act[0];   // gradient copy of the FC2 stage (read by dW_fc2)
    void* const g1 = sc.g_act[1];   // ... of the output-projection stage (read by dW_o)
    for (int i = d.nb - 1; i >= 0; --i) {
      const BlockSaved& s = sv[i];
      const sr_block_params& w = p[i];
      const sr_block_grads& g = gr[i];
      const int par = i & 1;
      void* const dz = sc.dz[par];
      void* const dqkv = sc.dqkv[par];
      ReduceJob jobs[6];   // this block's reductions (weights, LN2, the previous LN1), after dW_qkv
      if (ada) {
        // MLP-branch gradient dm = dh' * gate2 (activation copy) and dgate2 = sum_s dh' * m_out
        SR_TRY(join(kFc2));   // g0 may still be read by the previous block's dW_fc2
        ProfScope ps("convert", 0, (double)M * D * (e + 4), st);
        SR_TRY(launch_convert(kF32, sc.g_res, d.dtype, g0, (size_t)M * D, s.mod + 5 * D, 6 * D, S, D, nullptr, st));
        SR_TRY(gate_grad(d, sc.g_res, s.m_out, sc.dmod, 5 * D, sc, st));
      }
      // FC2: dW2, db2; dz = (dm W2) * GELU'(z)
      SR_TRY(on_side(kFc2, [&](hipStream_t ss) -> hipError_t {
        if (g.w_fc2 || g.b_fc2) {   // GELU(z) recomputed from the stored pre-activation
          ProfScope ps("recompute", 0, (double)M * F * e * 2, ss);
          SR_TRY(launch_gelu(d.dtype, s.z, sc.gz_rc, (size_t)M * F, ss));
        }
        return weight_grad("gemm_dw_fc2", d, g0, D, sc.gz_rc, F, g.w_fc2, g.b_fc2, sc, kWgFc2, &jobs[kWgFc2], ss);
      }));
      SR_TRY(join(kFc1 + par));   // dz[par] may still be read by dW_fc1 two blocks back
      {
        GemmDesc gd = desc(d, g0, true, D, (size_t)M * D * e, w.w_fc2, false, F, (size_t)D * F * e, M, F, D);
        EpiArgs ep; ep.z_in = s.z; ep.out_act = dz; ep.ldo = F;
        SR_TRY(fork_point([&]() -> hipError_t {
          ProfScope ps("gemm_dx_fc2", gemm_flops(M, F, D), gemm_bytes(d, M, F, D, 2 * (int)e), st);
          return launch_gemm(gd, EPI_DGELU, ep, st);
        }));
      }
      // FC1: dW1, db1; du = dz W1
      SR_TRY(on_side(kFc1 + par, [&](hipStream_t ss) -> hipError_t {
        if (g.w_fc1 || g.b_fc1) {   // u2 = LN2(h1) recomputed from the saved statistics
          ProfScope ps("recompute", 0, (double)M * D * (4 + e), ss);
          SR_TRY(launch_ln_apply(d.dtype, s.h1, w.ln2_w, w.ln2_b, ada ? s.mod : nullptr, 3 * D, M, S, D, s.mean2,
                                 s.rstd2, sc.u_rc, ss));
        }
        return weight_grad("gemm_dw_fc1", d, dz, F, sc.u_rc, D, g.w_fc1, g.b_fc1, sc, kWgFc1, &jobs[kWgFc1], ss);
      }));
      {
        GemmDesc gd = desc(d, dz, true, F, (size_t)M * F * e, w.w_fc1, false, D, (size_t)F * D * e, M, D, F);
        EpiArgs ep; ep.out_f32 = sc.du; ep.ldo = D;
        ProfScope ps("gemm_dx_fc1", gemm_flops(M, D, F), gemm_bytes(d, M, D, F, 4), st);
        SR_TRY(launch_gemm(gd, EPI_F32, ep, st));
      }
      // LN2 backward: g_res2 = g_res + LN2^T du (pre-LN also writes the activation copy)
      if (!ada) SR_TRY(join(kO));   // g1 may still be read by the previous block's dW_o
      SR_TRY(fork_point([&]() -> hipError_t {
        ProfScope ps("ln_bwd", 0, (double)M * D * (16 + e), st);
        return launch_ln_bwd(d.dtype, sc.du, s.h1, s.mean2, s.rstd2, w.ln2_w, ada ? s.mod : nullptr, 3 * D, sc.g_res,
                             d.B, S, D, sc.g_res2, ada ? nullptr : g1, sc.lnpart[0][ada ? 0 : par], st);
      }));
      if (ada) {   // dscale2 -> dmod[4D..5D), dshift2 -> dmod[3D..4D)
        ProfScope ps("reduce", 0, (double)d.B * nln * 2 * D * 4, st);
        SR_TRY(launch_reduce_cols(sc.lnpart[0][0], nln, d.B, 0, 2 * D, D, sc.dmod + 4 * D, sc.dmod + 3 * D, 6 * D,
                                  st));
      }
      if (ada) {
        // attention-branch gradient da = dh1 * gate1 and dgate1 = sum_s dh1 * a_out
        SR_TRY(gate_grad(d, sc.g_res2, s.a_out, sc.dmod, 2 * D, sc, st));
        SR_TRY(join(kO));   // g1 may still be read by the previous block's dW_o
        ProfScope ps("convert", 0, (double)M * D * (e + 4), st);
        SR_TRY(launch_convert(kF32, sc.g_res2, d.dtype, g1, (size_t)M * D, s.mod + 2 * D, 6 * D, S, D, nullptr, st));
      }
      // output projection: dWo, dbo; dO = da Wo (with the attention row statistic
      // delta = rowsum(dO * O) per head in the same epilogue when the head dim is 64)
      SR_TRY(on_side(kO, [&](hipStream_t ss) -> hipError_t {
        return weight_grad("gemm_dw_o", d, g1, D, s.O, D, g.w_o, g.b_o, sc, kWgO, &jobs[kWgO], ss);
      }));
      const bool fuse_delta = d.dtype == kBF16 && D / d.H == 64;
      {
        GemmDesc gd = desc(d, g1, true, D, (size_t)M * D * e, w.w_o, false, D, (size_t)D * D * e, M, D, D);
        EpiArgs ep; ep.out_act = sc.dO; ep.ldo = D;
        ep.o_in = s.O; ep.delta = sc.delta; ep.S = S; ep.H = d.H;
        ProfScope ps("gemm_dx_o", gemm_flops(M, D, D), gemm_bytes(d, M, D, D, (int)e), st);
        SR_TRY(launch_gemm(gd, fuse_delta ? EPI_DO : EPI_ACT, ep, st));
      }
      // attention backward
      if (!fuse_delta) {
        ProfScope ps("attn_bwd_delta", 0, (double)M * D * e * 2, st);
        SR_TRY(launch_attn_delta(d.dtype, sc.dO, s.O, d.B, S, d.H, D / d.H, sc.delta, st));
      }
      SR_TRY(join(kQkv + par));   // dqkv[par] may still be read by dW_qkv two blocks back
      SR_TRY(fork_point([&]() -> hipError_t {
        return launch_attn_bwd(d.dtype, s.qkv, sc.dO, s.lse, sc.delta, dqkv, d.B, S, d.H, D, st);
      }));
      if (!ada) {   // LN2 of this block and LN1 of the block before it join the reduction launch
        if (g.ln2_w || g.ln2_b) jobs[4] = ln_job(sc.lnpart[0][par], g.ln2_w, g.ln2_b);
        if (ln1_pending && (ln1_pending->ln1_w || ln1_pending->ln1_b))
          jobs[5] = ln_job(ln1_pending_part, ln1_pending->ln1_w, ln1_pending->ln1_b);
      }
      // QKV: dWqkv, dbqkv; du = dqkv Wqkv
      SR_TRY(on_side(kQkv + par, [&](hipStream_t ss) -> hipError_t {
        if (g.w_qkv || g.b_qkv) {   // u1 = LN1(h) recomputed from the saved statistics
          ProfScope ps("recompute", 0, (double)M * D * (4 + e), ss);
          SR_TRY(launch_ln_apply(d.dtype, s.hin, w.ln1_w, w.ln1_b, ada ? s.mod : nullptr, 0, M, S, D, s.mean1,
                                 s.rstd1, sc.u_rc, ss));
        }
        SR_TRY(weight_grad("gemm_dw_qkv", d, dqkv, 3 * D, sc.u_rc, D, g.w_qkv, g.b_qkv, sc, kWgQkv, &jobs[kWgQkv],
                           ss));
        // the block's reductions in one launch, each in the order of its single kernel
        ProfScope ps("reduce_dw", 0, 0, ss);
        return launch_reduce_jobs(jobs, 6, ss);
      }));
      ln1_pending = nullptr;
      {
        GemmDesc gd = desc(d, dqkv, true, 3 * D, (size_t)M * 3 * D * e, w.w_qkv, false, D, (size_t)3 * D * D * e,
                           M, D, 3 * D);
        EpiArgs ep; ep.out_f32 = sc.du; ep.ldo = D;
        ProfScope ps("gemm_dx_qkv", gemm_flops(M, D, 3 * D), gemm_bytes(d, M, D, 3 * D, 4), st);
        SR_TRY(launch_gemm(gd, EPI_F32, ep, st));
      }
      // LN1 backward: g_res = g_res2 + LN1^T du (pre-LN: plus the activation copy for the next block)
      if (!ada) SR_TRY(join(kFc2));   // g0 is still read by this block's dW_fc2
      SR_TRY(fork_point([&]() -> hipError_t {
        ProfScope ps("ln_bwd", 0, (double)M * D * (16 + e), st);
        return launch_ln_bwd(d.dtype, sc.du, s.hin, s.mean1, s.rstd1, w.ln1_w, ada ? s.mod : nullptr, 0, sc.g_res2,
                             d.B, S, D, sc.g_res, ada ? nullptr : g0, sc.lnpart[ada ? 0 : 1][ada ? 0 : par], st);
      }));
      if (ada) {   // dscale1 -> dmod[D..2D), dshift1 -> dmod[0..D)
        ProfScope ps("reduce", 0, (double)d.B * nln * 2 * D * 4, st);
        SR_TRY(launch_reduce_cols(sc.lnpart[0][0], nln, d.B, 0, 2 * D, D, sc.dmod + D, sc.dmod, 6 * D, st));
      } else {
        ln1_pending = &g;
        ln1_pending_part = sc.lnpart[1][par];
      }
      if (ada) {
        // dW_ada = dmod^T c ; db_ada = sum_b dmod ; dcond (+)= dmod W_ada
        ProfScope ps("mod", 0, 0, st);
        if (g.w_ada) {
          GemmDesc gd = desc(d, sc.dmod, false, 6 * D, (size_t)d.B * 6 * D * 4, cond, false, D, (size_t)d.B * D * e,
                             6 * D, D, d.B);
          gd.use_mfma = false; gd.a_type = kF32;
          EpiArgs ep; ep.out_f32 = g.w_ada; ep.ldo = D;
          SR_TRY(launch_gemm(gd, EPI_F32, ep, st));
        }
        if (g.b_ada) SR_TRY(launch_reduce_cols(sc.dmod, d.B, 1, 1, 6 * D, 6 * D, g.b_ada, nullptr, 0, st));
        if (dcond)   // dcond (+)= dmod W_ada, summed over the blocks in backward order
          SR_TRY(launch_gemv_cols(d.dtype, sc.dmod, 6 * D, w.w_ada, d.B, 6 * D, D, dcond, i == d.nb - 1 ? 0 : 1,
                                  sc.gvpart, st));
        // parameters the adaLN block does not use get zero gradients
        SR_TRY(zero_f32(g.ln1_w, D, st)); SR_TRY(zero_f32(g.ln1_b, D, st));
        SR_TRY(zero_f32(g.ln2_w, D, st)); SR_TRY(zero_f32(g.ln2_b, D, st));
      } else {
        SR_TRY(zero_f32(g.w_ada, (size_t)6 * D * D, st));
        SR_TRY(zero_f32(g.b_ada, (size_t)6 * D, st));
      }
    }
    if (rt) {   // residual-delta scatter of the gradient fused with its rounding
      ProfScope ps("scatter_f32", 0, (double)M * D * (2 * e + 4) + 4.0 * M, st);
      SR_TRY(launch_scatter_f32_delta(d.dtype, d.B, d.L, S, D, rt->x, sc.g_res, rt->idx, rt->shared, st));
    } else {
      ProfScope ps("convert", 0, (double)M * D * (e + 4), st);
      SR_TRY(launch_convert(kF32, sc.g_res, d.dtype, dh_in, (size_t)M * D, nullptr, 0, S, D, nullptr, st));
    }
    if (ln1_pending && (ln1_pending->ln1_w || ln1_pending->ln1_b)) {
      ProfScope ps("reduce", 0, (double)d.B * nln * 2 * D * 4, st);
      SR_TRY(launch_reduce_cols(ln1_pending_part, nln, d.B, 1, 2 * D, D, ln1_pending->ln1_w, ln1_pending->ln1_b, 0,
                                st));
    }
    for (int k = 0; k < kSlots; ++k) SR_TRY(join(k));   // every gradient is complete when st is
    return hipSuccess;
  };
  hipError_t err = run();
  if (err != hipSuccess && side && ev) {
    // leave no weight-gradient work unordered with respect to the caller's stream
    for (int k = 0; k < kSlots; ++k)
      if (pending[k]) (void)hipStreamWaitEvent(st, ev->done[k], 0);
  }
  give_events(ev);
  delete[] sv;
  return err;
}

}  // namespace sr
