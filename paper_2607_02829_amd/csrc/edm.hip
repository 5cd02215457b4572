// The generative model's block with the asymmetric attention of the sparse middle stage
// (Sec. 3.4 "Integration with Generative Forecasting", Alg. 2 stage 2; Sec. 3.1 "Generative
// forecasting"; App. A.1 EDM table), forward and backward, as launch sequences over the
// library's GEMM, LayerNorm, GEMV and attention kernels.
//
// Per block, with e the noise embedding [B, D] and Z_c the conditioning tokens [B, L, D]:
//   (shift, scale) = e W_film^T + b_film           gemv rows -> mod[:, 0:2D]
//   g = sigmoid(e W_g^T + b_g)                     gemv rows -> mod[:, 2D:3D], sigmoid in place
//   u  = LN0(h) (1 + scale) + shift                ln_fwd with modulation (no affine)
//   qkv = u W_qkv^T + b_qkv; O = SelfAttn(qkv)     gemm, attention over the S tokens
//   h1 = h + O W_o^T + b_o                         gemm, residual epilogue (fp32 stream)
//   uc = LNc(h1); qc = uc W_q^T + b_q              ln_fwd (affine), gemm
//   kvc = Z_c W_kv^T + b_kv                        gemm over the B L conditioning rows
//   Oc = CrossAttn(qc, kvc)                        attention, S queries x L keys
//   h2 = h1 + g (Oc W_oc^T + b_oc)                 gemm, gated residual epilogue (saves c_out)
//   h' = h2 + MLP(LN2(h2))                         as the pre-LN block
// The S tokens are the K routed ones in the sparse stage (S = L for the dense block); the
// conditioning keeps its L tokens, so the cross-attention costs O(S L D).  The modulation row
// of a sample holds (shift, scale, gate) at columns 0, D, 2D of a 6D row, the layout the
// modulated LayerNorm kernels read.
//
// Backward: the vector-Jacobian products in reverse order; the gate's logit gradient is
// sum_s (dh2 c_out) g (1 - g); Z_c's gradient is the sum over blocks of dkvc W_kv and e's the
// sum over blocks of dfilm W_film + dlogit W_g.  Every launch is on the caller's stream.
#include "edm.h"

#include <algorithm>
#include <cmath>
#include <vector>

#include "common.h"
#include "profile.h"

namespace sr {

namespace {

#define SR_TRY(x)                    \
  do {                               \
    hipError_t _e = (x);             \
    if (_e != hipSuccess) return _e; \
  } while (0)

// ------------------------------------------------------------------------------ kernels

// mod[b * ld + c] <- sigmoid(mod[b * ld + c]) for c < D: the sigma-gate.
__global__ __launch_bounds__(256) void sigmoid_kernel(float* __restrict__ x, int B, int D, int ld) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * D) return;
  float* p = x + (size_t)(i / D) * ld + i % D;
  *p = 1.0f / (1.0f + expf(-*p));
}

// d[b * ld + c] *= g (1 - g), g = gate[b * ld + c]: from the gradient of the gate to that of its
// logit.
__global__ __launch_bounds__(256) void sigmoid_grad_kernel(float* __restrict__ d, const float* __restrict__ gate,
                                                           int B, int D, int ld) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= B * D) return;
  const size_t o = (size_t)(i / D) * ld + i % D;
  const float g = gate[o];
  d[o] *= g * (1.0f - g);
}

// out[c] = sum over b (ascending) of x[b * ld + c], c < n: the bias gradients of the per-sample
// modulation (few samples).
__global__ __launch_bounds__(256) void sum_samples_kernel(const float* __restrict__ x, int B, int n, int ld,
                                                          float* __restrict__ out) {
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= n) return;
  float s = 0.f;
  for (int b = 0; b < B; ++b) s += x[(size_t)b * ld + c];
  out[c] = s;
}

hipError_t launch_sigmoid(float* x, int B, int D, int ld, hipStream_t st) {
  SR_LAUNCH(sigmoid_kernel, dim3((B * D + 255) / 256), dim3(256), 0, st, x, B, D, ld);
  return hipGetLastError();
}
hipError_t launch_sigmoid_grad(float* d, const float* gate, int B, int D, int ld, hipStream_t st) {
  SR_LAUNCH(sigmoid_grad_kernel, dim3((B * D + 255) / 256), dim3(256), 0, st, d, gate, B, D, ld);
  return hipGetLastError();
}
hipError_t launch_sum_samples(const float* x, int B, int n, int ld, float* out, hipStream_t st) {
  if (!out) return hipSuccess;
  SR_LAUNCH(sum_samples_kernel, dim3((n + 255) / 256), dim3(256), 0, st, x, B, n, ld, out);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------ host helpers

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

double gflops(double M, double N, double K) { return 2.0 * M * N * K; }

GemmDesc desc(const EdmDims& d, const void* A, bool ak, long long lda, size_t abytes, const void* B, bool bk,
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

// Y[rows, N] = X[rows, K] W^T + bias (X and W storage type, nn.Linear W [N, K]), epilogue epi.
hipError_t linear(const char* name, const EdmDims& d, const void* X, int rows, int K, const void* W, int N, int epi,
                  const EpiArgs& ep, hipStream_t st) {
  GemmDesc g = desc(d, X, true, K, (size_t)rows * K * d.elt, W, true, K, (size_t)N * K * d.elt, rows, N, K);
  ProfScope ps(name, gflops(rows, N, K), ((double)rows * K + (double)N * K + (double)rows * N) * d.elt, st);
  return launch_gemm(g, epi, ep, st);
}

// dX[rows, K] = dY[rows, N] W (W [N, K]), epilogue epi.
hipError_t linear_dx(const char* name, const EdmDims& d, const void* dY, int rows, int N, const void* W, int K,
                     int epi, const EpiArgs& ep, hipStream_t st) {
  GemmDesc g = desc(d, dY, true, N, (size_t)rows * N * d.elt, W, false, K, (size_t)N * K * d.elt, rows, K, N);
  ProfScope ps(name, gflops(rows, K, N), ((double)rows * N + (double)N * K) * d.elt + (double)rows * K * 4, st);
  return launch_gemm(g, epi, ep, st);
}

// dW[N, K] = dY^T X and db[N] = column sums of dY, over `rows` tokens (both token-major).
hipError_t wgrad(const char* name, const EdmDims& d, const void* dY, int N, const void* X, int K, int rows, float* dw,
                 float* db, const EdmScratch& sc, hipStream_t st) {
  if (!dw && !db) return hipSuccess;
  GemmDesc g = desc(d, dY, false, N, (size_t)rows * N * d.elt, X, false, K, (size_t)rows * K * d.elt, N, K, rows);
  size_t pf = 0, df = 0;
  if (g.use_mfma) weight_grad_scratch(N, K, rows, &pf, &df);
  float* out = dw ? dw : sc.wpart + pf;   // the kernel always produces dW; park an unwanted one
  ProfScope ps(name, gflops(N, K, rows), ((double)rows * (N + K)) * d.elt + (double)N * K * 4, st);
  return launch_weight_grad(g, out, db, sc.wpart, sc.dbpart, st);
}


}  // namespace

size_t edm_layout_saved(const EdmDims& d, char* base, EdmSaved* out) {
  Carver c(base);
  const size_t M = d.M, Mc = d.Mc, D = d.D, F = d.F, e = d.elt;
  const size_t stats = (size_t)d.B * d.H * d.S * 4;
  for (int i = 0; i < d.nb; ++i) {
    EdmSaved s{};
    s.mod = c.take<float>((size_t)d.B * 6 * D * 4);
    s.hin = c.take<float>(M * D * 4);
    s.mean0 = c.take<float>(M * 4);
    s.rstd0 = c.take<float>(M * 4);
    s.u = c.take<void>(M * D * e);
    s.qkv = c.take<void>(M * 3 * D * e);
    s.O = c.take<void>(M * D * e);
    s.lse = c.take<float>(stats);
    s.h1 = c.take<float>(M * D * 4);
    s.meanc = c.take<float>(M * 4);
    s.rstdc = c.take<float>(M * 4);
    s.uc = c.take<void>(M * D * e);
    s.qc = c.take<void>(M * D * e);
    s.kvc = c.take<void>(Mc * 2 * D * e);
    s.Oc = c.take<void>(M * D * e);
    s.lsec = c.take<float>(stats);
    s.c_out = c.take<void>(M * D * e);
    s.h2 = c.take<float>(M * D * 4);
    s.mean2 = c.take<float>(M * 4);
    s.rstd2 = c.take<float>(M * 4);
    s.u2 = c.take<void>(M * D * e);
    s.z = c.take<void>(M * F * e);
    s.gz = c.take<void>(M * F * e);
    if (out) out[i] = s;
  }
  return c.off;
}

size_t edm_layout_scratch(const EdmDims& d, char* base, EdmScratch* out) {
  Carver c(base);
  const size_t M = d.M, Mc = d.Mc, D = d.D, F = d.F, e = d.elt;
  EdmScratch s{};
  s.g_res = c.take<float>(M * D * 4);
  s.g_res2 = c.take<float>(M * D * 4);
  s.du = c.take<float>(M * D * 4);
  s.delta = c.take<float>((size_t)d.B * d.H * d.S * 4);
  // weight-gradient scratch: split partials of the largest case, plus room for an unwanted dW
  size_t wp = 0, dbp = 0, wout = 0;
  // (rows of dW, columns of dW, tokens reduced): W_qkv; W_o, W_oc, W_q; W_fc1; W_fc2; W_kv
  const int shapes[5][3] = {{3 * d.D, d.D, d.M}, {d.D, d.D, d.M}, {d.F, d.D, d.M}, {d.D, d.F, d.M},
                            {2 * d.D, d.D, d.Mc}};
  for (const auto& sh : shapes) {
    size_t pf = 0, df = 0;
    if (d.dtype == kBF16) weight_grad_scratch(sh[0], sh[1], sh[2], &pf, &df);
    wp = std::max(wp, pf);
    dbp = std::max(dbp, df);
    wout = std::max(wout, (size_t)sh[0] * sh[1]);
  }
  s.wpart = c.take<float>((wp + wout) * 4);
  s.dbpart = c.take<float>(std::max<size_t>(dbp, 1) * 4);
  s.part = c.take<float>((size_t)d.B * colsum_chunks(d.S) * D * 4);
  s.lnpart = c.take<float>((size_t)d.B * ln_bwd_chunks(d.S) * 2 * D * 4);
  s.dmod = c.take<float>((size_t)d.B * 6 * D * 4);
  s.gvpart = c.take<float>(std::max(gemv_cols_scratch(d.B, 2 * d.D, d.D), gemv_cols_scratch(d.B, d.D, d.D)) * 4);
  s.g_act = c.take<void>(M * D * e);
  s.dc = c.take<void>(M * D * e);
  s.dz = c.take<void>(M * F * e);
  s.dO = c.take<void>(M * D * e);
  s.dqkv = c.take<void>(M * 3 * D * e);
  s.dqc = c.take<void>(M * D * e);
  s.dkvc = c.take<void>(Mc * 2 * D * e);
  if (out) *out = s;
  return c.off;
}

// ============================================================================ forward

hipError_t edm_fwd(const EdmDims& d, const sr_edm_block_params* p, const void* e_sig, const void* zc,
                   const void* h_in, void* h_out, char* saved, hipStream_t st) {
  std::vector<EdmSaved> sv((size_t)d.nb);
  edm_layout_saved(d, saved, sv.data());
  const int M = d.M, Mc = d.Mc, D = d.D, F = d.F, S = d.S, B = d.B;
  {
    ProfScope ps("convert", 0, (double)M * D * (d.elt + 4), st);
    SR_TRY(launch_convert(d.dtype, h_in, kF32, sv[0].hin, (size_t)M * D, nullptr, 0, S, D, nullptr, st));
  }
  for (int i = 0; i < d.nb; ++i) {
    const EdmSaved& s = sv[(size_t)i];
    const sr_edm_block_params& w = p[i];
    {   // FiLM (shift, scale) and the sigma-gate from the noise embedding
      ProfScope ps("mod", gflops(B, 3 * D, D), (double)3 * D * D * d.elt, st);
      SR_TRY(launch_gemv_rows(d.dtype, e_sig, D, w.w_film, w.b_film, B, 2 * D, D, s.mod, 6 * D, st));
      SR_TRY(launch_gemv_rows(d.dtype, e_sig, D, w.w_g, w.b_g, B, D, D, s.mod + 2 * D, 6 * D, st));
      SR_TRY(launch_sigmoid(s.mod + 2 * D, B, D, 6 * D, st));
    }
    {
      ProfScope ps("ln_fwd", 0, (double)M * D * (4 + d.elt), st);
      SR_TRY(launch_ln_fwd(d.dtype, s.hin, nullptr, nullptr, s.mod, 0, M, S, D, d.eps, s.u, s.mean0, s.rstd0, st));
    }
    {
      EpiArgs ep; ep.out_act = s.qkv; ep.bias = w.b_qkv; ep.ldo = 3 * D;
      SR_TRY(linear("gemm_qkv", d, s.u, M, D, w.w_qkv, 3 * D, EPI_BIAS_ACT, ep, st));
    }
    {
      ProfScope ps("attn_fwd", 4.0 * B * (double)S * S * D, (double)M * D * d.elt * 4, st);
      SR_TRY(launch_attn_fwd(d.dtype, s.qkv, s.O, s.lse, B, S, d.H, D, st));
    }
    {
      EpiArgs ep; ep.bias = w.b_o; ep.resid = s.hin; ep.out_f32 = s.h1; ep.ldo = D; ep.S = S;
      SR_TRY(linear("gemm_o", d, s.O, M, D, w.w_o, D, EPI_RESID, ep, st));
    }
    {
      ProfScope ps("ln_fwd", 0, (double)M * D * (4 + d.elt), st);
      SR_TRY(launch_ln_fwd(d.dtype, s.h1, w.lnc_w, w.lnc_b, nullptr, 0, M, S, D, d.eps, s.uc, s.meanc, s.rstdc, st));
    }
    {
      EpiArgs ep; ep.out_act = s.qc; ep.bias = w.b_q; ep.ldo = D;
      SR_TRY(linear("gemm_q", d, s.uc, M, D, w.w_q, D, EPI_BIAS_ACT, ep, st));
    }
    {   // keys and values of all L conditioning tokens
      EpiArgs ep; ep.out_act = s.kvc; ep.bias = w.b_kv; ep.ldo = 2 * D;
      SR_TRY(linear("gemm_kv", d, zc, Mc, D, w.w_kv, 2 * D, EPI_BIAS_ACT, ep, st));
    }
    {
      ProfScope ps("xattn_fwd", 4.0 * B * (double)S * d.L * D, (double)B * (2.0 * S + 2.0 * d.L) * D * d.elt, st);
      SR_TRY(launch_xattn_fwd(d.dtype, s.qc, s.kvc, s.Oc, s.lsec, B, S, d.L, d.H, D, st));
    }
    {   // h2 = h1 + g (Oc W_oc^T + b_oc); the ungated branch is saved for the gate's gradient
      EpiArgs ep; ep.bias = w.b_oc; ep.resid = s.h1; ep.out_f32 = s.h2; ep.ldo = D; ep.S = S;
      ep.gate = s.mod + 2 * D; ep.gate_stride = 6 * D; ep.a_save = s.c_out;
      SR_TRY(linear("gemm_oc", d, s.Oc, M, D, w.w_oc, D, EPI_RESID, ep, st));
    }
    {
      ProfScope ps("ln_fwd", 0, (double)M * D * (4 + d.elt), st);
      SR_TRY(launch_ln_fwd(d.dtype, s.h2, w.ln2_w, w.ln2_b, nullptr, 0, M, S, D, d.eps, s.u2, s.mean2, s.rstd2, st));
    }
    {
      EpiArgs ep; ep.bias = w.b_fc1; ep.out_act = s.z; ep.out_act2 = s.gz; ep.ldo = F;
      SR_TRY(linear("gemm_fc1", d, s.u2, M, D, w.w_fc1, F, EPI_GELU, ep, st));
    }
    {
      EpiArgs ep; ep.bias = w.b_fc2; ep.resid = s.h2; ep.ldo = D; ep.S = S;
      if (i + 1 < d.nb) ep.out_f32 = sv[(size_t)i + 1].hin;
      else ep.out_st = h_out;
      SR_TRY(linear("gemm_fc2", d, s.gz, M, F, w.w_fc2, D, EPI_RESID, ep, st));
    }
  }
  return hipSuccess;
}

// ============================================================================ backward

hipError_t edm_bwd(const EdmDims& d, const sr_edm_block_params* p, const void* e_sig, const void* zc,
                   const char* saved, const void* dh_out, void* dh_in, const sr_edm_block_grads* gr, float* dzc,
                   float* de, char* scratch, hipStream_t st) {
  std::vector<EdmSaved> sv((size_t)d.nb);
  edm_layout_saved(d, const_cast<char*>(saved), sv.data());
  EdmScratch sc;
  edm_layout_scratch(d, scratch, &sc);
  const int M = d.M, Mc = d.Mc, D = d.D, F = d.F, S = d.S, B = d.B;
  const int nln = ln_bwd_chunks(S);
  auto reduce_ln = [&](float* dw, float* dbeta) -> hipError_t {
    if (!dw && !dbeta) return hipSuccess;
    ProfScope ps("reduce", 0, (double)B * nln * 2 * D * 4, st);
    return launch_reduce_cols(sc.lnpart, nln, B, 1, 2 * D, D, dw, dbeta, 0, st);
  };
  // The weight-gradient GEMMs run on the library's second stream, forked from st after their
  // inputs are written; st waits for one (join) before it overwrites a buffer that GEMM reads:
  // g_act (dW_fc2, then dW_o) within the block, dz, dc, dqc, dkvc and dqkv in the next block.
  // The GEMMs share the split-K partial buffers, which the second stream's order serialises.
  // While every launch group is being profiled they run on st, so each group's time is its own.
  enum { kFc2 = 0, kFc1 = 1, kOc = 2, kQ = 3, kKv = 4, kO = 5, kQkv = 6 };
  const bool serial = profiling_all();
  hipStream_t side = nullptr;
  BwdEvents* ev = nullptr;
  bool pending[kSlots] = {};
  // Fork points: the kernels right before a fork carry the fork event themselves (bound at
  // launch, see LaunchHook), and the fork waits on the event the last of them carries; a fork
  // that follows another with no kernel launched in between needs no wait at all (the second
  // stream is already ordered after that point).  Not while st is being captured into a graph.
  hipStreamCaptureStatus capture = hipStreamCaptureStatusNone;
  const bool bind = !serial && hipStreamIsCapturing(st, &capture) == hipSuccess &&
                    capture == hipStreamCaptureStatusNone;
  hipEvent_t fork_ev = nullptr;
  unsigned long long fork_at = 0, forked_at = ~0ull;
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
  auto on_side = [&](int slot, auto&& launch) -> hipError_t {
    if (serial) return launch(st);
    const unsigned long long now = launch_hook().launches;
    if (bind && now == forked_at) {
      // nothing launched since the previous fork: the second stream already waits for it
    } else if (fork_ev && now == fork_at) {
      SR_TRY(hipStreamWaitEvent(side, fork_ev, 0));
    } else {
      SR_TRY(hipEventRecord(ev->fork, st));
      SR_TRY(hipStreamWaitEvent(side, ev->fork, 0));
    }
    fork_ev = nullptr;
    SR_TRY(launch(side));
    SR_TRY(hipEventRecord(ev->done[slot], side));
    forked_at = launch_hook().launches;   // counts the second stream's launches too
    pending[slot] = true;
    return hipSuccess;
  };
  auto join = [&](int slot) -> hipError_t {
    if (pending[slot]) SR_TRY(hipStreamWaitEvent(st, ev->done[slot], 0));
    pending[slot] = false;
    return hipSuccess;
  };
  auto run = [&]() -> hipError_t {
  if (!serial) {
    SR_TRY(side_stream(&side));
    SR_TRY(take_events(&ev));
  }
  {   // g_res = fp32(dh_out) and its storage copy
    ProfScope ps("convert", 0, (double)M * D * (2 * d.elt + 4), st);
    SR_TRY(launch_convert(d.dtype, dh_out, d.dtype, sc.g_act, (size_t)M * D, nullptr, 0, S, D, sc.g_res, st));
  }
  for (int i = d.nb - 1; i >= 0; --i) {
    const EdmSaved& s = sv[(size_t)i];
    const sr_edm_block_params& w = p[i];
    const sr_edm_block_grads& g = gr[i];
    const bool first = i == d.nb - 1;   // the first block of the backward writes the shared sums
    // ---------------------------------------------------------------- MLP
    SR_TRY(on_side(kFc2, [&](hipStream_t ss) {
      return wgrad("gemm_dw_fc2", d, sc.g_act, D, s.gz, F, M, g.w_fc2, g.b_fc2, sc, ss);
    }));
    SR_TRY(join(kFc1));   // dz may still be read by the previous block's dW_fc1
    {
      EpiArgs ep; ep.z_in = s.z; ep.out_act = sc.dz; ep.ldo = F;
      SR_TRY(fork_point([&] { return linear_dx("gemm_dx_fc2", d, sc.g_act, M, D, w.w_fc2, F, EPI_DGELU, ep, st); }));
    }
    SR_TRY(on_side(kFc1, [&](hipStream_t ss) {
      return wgrad("gemm_dw_fc1", d, sc.dz, F, s.u2, D, M, g.w_fc1, g.b_fc1, sc, ss);
    }));
    {
      EpiArgs ep; ep.out_f32 = sc.du; ep.ldo = D;
      SR_TRY(linear_dx("gemm_dx_fc1", d, sc.dz, M, F, w.w_fc1, D, EPI_F32, ep, st));
    }
    {   // dh2 = dh' + LN2^T du
      ProfScope ps("ln_bwd", 0, (double)M * D * (16 + d.elt), st);
      SR_TRY(launch_ln_bwd(d.dtype, sc.du, s.h2, s.mean2, s.rstd2, w.ln2_w, nullptr, 0, sc.g_res, B, S, D, sc.g_res2,
                           nullptr, sc.lnpart, st));
    }
    SR_TRY(reduce_ln(g.ln2_w, g.ln2_b));
    // ---------------------------------------------------------------- gated cross-attention
    SR_TRY(join(kOc));   // dc may still be read by the previous block's dW_oc
    {   // dc = dh2 g (storage copy); dlogit = sum_s dh2 c_out, then times g (1 - g)
      ProfScope ps("convert", 0, (double)M * D * (d.elt + 4), st);
      SR_TRY(launch_convert(kF32, sc.g_res2, d.dtype, sc.dc, (size_t)M * D, s.mod + 2 * D, 6 * D, S, D, nullptr, st));
    }
    SR_TRY(fork_point([&]() -> hipError_t {
      ProfScope ps("colsum", 0, (double)M * D * (4 + d.elt), st);
      SR_TRY(launch_colsum(kF32, sc.g_res2, d.dtype, s.c_out, nullptr, 0, B, S, D, sc.part, st));
      SR_TRY(launch_reduce_cols(sc.part, colsum_chunks(S), B, 0, D, D, sc.dmod + 2 * D, nullptr, 6 * D, st));
      return launch_sigmoid_grad(sc.dmod + 2 * D, s.mod + 2 * D, B, D, 6 * D, st);
    }));
    SR_TRY(on_side(kOc, [&](hipStream_t ss) {
      return wgrad("gemm_dw_oc", d, sc.dc, D, s.Oc, D, M, g.w_oc, g.b_oc, sc, ss);
    }));
    {
      EpiArgs ep; ep.out_act = sc.dO; ep.ldo = D;
      SR_TRY(linear_dx("gemm_dx_oc", d, sc.dc, M, D, w.w_oc, D, EPI_ACT, ep, st));
    }
    SR_TRY(join(kQ));    // dqc and dkvc may still be read by the previous block's dW_q, dW_kv
    SR_TRY(join(kKv));
    {
      ProfScope ps("xattn_bwd", 8.0 * B * (double)S * d.L * D, (double)B * (5.0 * S + 4.0 * d.L) * D * d.elt, st);
      SR_TRY(fork_point([&] {
        return launch_xattn_bwd(d.dtype, s.qc, s.kvc, s.Oc, sc.dO, s.lsec, sc.delta, sc.dqc, sc.dkvc, B, S, d.L, d.H,
                                D, st);
      }));
    }
    SR_TRY(on_side(kQ, [&](hipStream_t ss) {
      return wgrad("gemm_dw_q", d, sc.dqc, D, s.uc, D, M, g.w_q, g.b_q, sc, ss);
    }));
    SR_TRY(on_side(kKv, [&](hipStream_t ss) {
      return wgrad("gemm_dw_kv", d, sc.dkvc, 2 * D, zc, D, Mc, g.w_kv, g.b_kv, sc, ss);
    }));
    if (dzc) {   // dZ_c (+)= dkvc W_kv, summed over the blocks in backward order
      EpiArgs ep; ep.out_f32 = dzc; ep.ldo = D;
      SR_TRY(linear_dx("gemm_dzc", d, sc.dkvc, Mc, 2 * D, w.w_kv, D, first ? EPI_F32 : EPI_F32_ACC, ep, st));
    }
    {
      EpiArgs ep; ep.out_f32 = sc.du; ep.ldo = D;
      SR_TRY(linear_dx("gemm_dx_q", d, sc.dqc, M, D, w.w_q, D, EPI_F32, ep, st));
    }
    SR_TRY(join(kFc2));   // g_act is still read by this block's dW_fc2
    {   // dh1 = dh2 + LNc^T duc, with its storage copy for the output projection
      ProfScope ps("ln_bwd", 0, (double)M * D * (16 + d.elt), st);
      SR_TRY(launch_ln_bwd(d.dtype, sc.du, s.h1, s.meanc, s.rstdc, w.lnc_w, nullptr, 0, sc.g_res2, B, S, D, sc.g_res,
                           sc.g_act, sc.lnpart, st));
    }
    SR_TRY(reduce_ln(g.lnc_w, g.lnc_b));
    // ---------------------------------------------------------------- FiLM-modulated self-attention
    SR_TRY(on_side(kO, [&](hipStream_t ss) {
      return wgrad("gemm_dw_o", d, sc.g_act, D, s.O, D, M, g.w_o, g.b_o, sc, ss);
    }));
    const bool fuse_delta = d.dtype == kBF16 && D / d.H == 64;
    {
      EpiArgs ep; ep.out_act = sc.dO; ep.ldo = D; ep.o_in = s.O; ep.delta = sc.delta; ep.S = S; ep.H = d.H;
      SR_TRY(linear_dx("gemm_dx_o", d, sc.g_act, M, D, w.w_o, D, fuse_delta ? EPI_DO : EPI_ACT, ep, st));
    }
    if (!fuse_delta) {
      ProfScope ps("attn_bwd_delta", 0, (double)M * D * d.elt * 2, st);
      SR_TRY(launch_attn_delta(d.dtype, sc.dO, s.O, B, S, d.H, D / d.H, sc.delta, st));
    }
    SR_TRY(join(kQkv));   // dqkv may still be read by the previous block's dW_qkv
    SR_TRY(fork_point([&] { return launch_attn_bwd(d.dtype, s.qkv, sc.dO, s.lse, sc.delta, sc.dqkv, B, S, d.H, D, st); }));
    SR_TRY(on_side(kQkv, [&](hipStream_t ss) {
      return wgrad("gemm_dw_qkv", d, sc.dqkv, 3 * D, s.u, D, M, g.w_qkv, g.b_qkv, sc, ss);
    }));
    {
      EpiArgs ep; ep.out_f32 = sc.du; ep.ldo = D;
      SR_TRY(linear_dx("gemm_dx_qkv", d, sc.dqkv, M, 3 * D, w.w_qkv, D, EPI_F32, ep, st));
    }
    SR_TRY(join(kO));   // g_act is still read by this block's dW_o
    {   // dh = dh1 + LN0^T (du (1 + scale)); its partial column sums give dshift, dscale
      ProfScope ps("ln_bwd", 0, (double)M * D * (16 + d.elt), st);
      SR_TRY(launch_ln_bwd(d.dtype, sc.du, s.hin, s.mean0, s.rstd0, nullptr, s.mod, 0, sc.g_res, B, S, D, sc.g_res2,
                           sc.g_act, sc.lnpart, st));
      SR_TRY(launch_reduce_cols(sc.lnpart, nln, B, 0, 2 * D, D, sc.dmod + D, sc.dmod, 6 * D, st));
    }
    std::swap(sc.g_res, sc.g_res2);   // the next block's output gradient
    {   // parameters of the modulation and the noise embedding's gradient
      ProfScope ps("mod", 0, 0, st);
      if (g.w_film) {   // dW_film = dfilm^T e (dfilm = dmod[:, 0:2D])
        GemmDesc gd = desc(d, sc.dmod, false, 6 * D, (size_t)B * 6 * D * 4, e_sig, false, D, (size_t)B * D * d.elt,
                           2 * D, D, B);
        gd.use_mfma = false; gd.a_type = kF32;
        EpiArgs ep; ep.out_f32 = g.w_film; ep.ldo = D;
        SR_TRY(launch_gemm(gd, EPI_F32, ep, st));
      }
      if (g.w_g) {      // dW_g = dlogit^T e (dlogit = dmod[:, 2D:3D])
        GemmDesc gd = desc(d, sc.dmod + 2 * D, false, 6 * D, (size_t)B * 6 * D * 4 - 2 * D * 4, e_sig, false, D,
                           (size_t)B * D * d.elt, D, D, B);
        gd.use_mfma = false; gd.a_type = kF32;
        EpiArgs ep; ep.out_f32 = g.w_g; ep.ldo = D;
        SR_TRY(launch_gemm(gd, EPI_F32, ep, st));
      }
      SR_TRY(launch_sum_samples(sc.dmod, B, 2 * D, 6 * D, g.b_film, st));
      SR_TRY(launch_sum_samples(sc.dmod + 2 * D, B, D, 6 * D, g.b_g, st));
      if (de) {   // de (+)= dfilm W_film + dlogit W_g, summed over the blocks in backward order
        SR_TRY(launch_gemv_cols(d.dtype, sc.dmod, 6 * D, w.w_film, B, 2 * D, D, de, first ? 0 : 1, sc.gvpart, st));
        SR_TRY(launch_gemv_cols(d.dtype, sc.dmod + 2 * D, 6 * D, w.w_g, B, D, D, de, 1, sc.gvpart, st));
      }
    }
  }
  {
    ProfScope ps("convert", 0, (double)M * D * (d.elt + 4), st);
    SR_TRY(launch_convert(kF32, sc.g_res, d.dtype, dh_in, (size_t)M * D, nullptr, 0, S, D, nullptr, st));
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
  return err;
}

}  // namespace sr
