// Internal interfaces of libsr: kernel launchers and the GEMM descriptor.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

namespace sr {

enum { kF32 = 0, kBF16 = 1 };

enum {
  EPI_BIAS_ACT = 0,
  EPI_RESID = 1,
  EPI_GELU = 2,
  EPI_DGELU = 3,
  EPI_ACT = 4,
  EPI_F32 = 5,
  EPI_F32_ACC = 6,
  EPI_BIAS_F32 = 7,
  EPI_DW = 8,
  EPI_DO = 9,   // dO store plus the attention row statistic delta (head dim 64)
};

struct EpiArgs {
  void* out_act = nullptr;     // activation-type output
  void* out_act2 = nullptr;    // second activation output (GELU value)
  float* out_f32 = nullptr;    // fp32 output
  void* out_st = nullptr;      // storage-type output
  const void* bias = nullptr;  // storage type, [N]
  const float* resid = nullptr;
  const float* gate = nullptr;  // per-sample column gate (adaLN), gate[b * gate_stride + n]
  int gate_stride = 0;
  void* a_save = nullptr;       // branch output saved before gating (adaLN)
  const void* z_in = nullptr;   // pre-activation for GELU'
  long long ldo = 0;            // row stride of the outputs
  int S = 1;                    // rows per sample (gate indexing)
  // EPI_RESID with sc_x: instead of out_st, the residual-delta scatter of the storage-rounded
  // result into the full sequence, x[b, i, n] = rnd(x0 + (rnd(r) - x0)), x0 = x[b, i, n],
  // i = sc_idx[(sc_shared ? 0 : b) * S + s] for row m = b * S + s (rows of x have ldo elements)
  void* sc_x = nullptr;
  const int32_t* sc_idx = nullptr;
  int sc_L = 0, sc_shared = 0;
  long long split_stride = 0;   // element stride between split-K partial outputs
  // EPI_DW (weight gradient, reduction over tokens): out_f32 receives dW and db_out (optional)
  // the row sums of A (the bias gradient); with split-K each split writes its plane of part,
  // and the bias-gradient sums are spread over the workgroups of a tile row (dbpart rows), so
  // launch_weight_grad adds the partial planes and rows in a fixed order.
  float* db_out = nullptr;
  float* part = nullptr;
  float* dbpart = nullptr;
  // EPI_DO: out_act = dO; delta[(b*H + h)*S + s] = sum over head h's 64 columns of
  // bf16(dO) * O, O read from o_in (token-major like dO)
  const void* o_in = nullptr;
  float* delta = nullptr;
  int H = 1;
};

struct GemmDesc {
  const void* A = nullptr;
  const void* B = nullptr;
  int M = 0, N = 0, K = 0;
  long long lda = 0, ldb = 0;
  size_t a_bytes = 0, b_bytes = 0;  // exact sizes of the operands (bounds of the buffer loads)
  bool a_kmajor = true, b_kmajor = true;
  int splits = 1, k_per_split = 0;
  bool use_mfma = false;
  int dtype = kBF16;          // storage type (bias / residual output)
  int a_type = kBF16, b_type = kBF16;
};

hipError_t launch_select_random(int rows, int L, int K, uint64_t seed, uint64_t step, int32_t* idx, hipStream_t st);
hipError_t launch_select_topk(int dtype, int rows, int L, int D, int K, const void* xt, const void* xp, float* score,
                              int32_t* idx, hipStream_t st);
// Allocation-free top-k selection: fp32 scores of at most kSelStaticScores tokens (rows * L) in a
// file-scope device array of select.hip; *out receives its address on the current device.
constexpr int kSelStaticScores = 1 << 20;
hipError_t select_static_scratch(float** out);
hipError_t launch_select_topk_planes(int rows, int L, int K, int parts, const float* planes, int32_t* idx,
                                     hipStream_t st);
hipError_t launch_validate(const int32_t* idx, int rows, int K, int L, int32_t* ok, hipStream_t st);

// The backward's second stream (one per device, default priority, kept for the life of the
// process) for the weight-gradient work, and pooled event sets of one backward call: fork
// (caller stream -> second stream) and, per slot, the completion of the last weight-gradient
// work that read a buffer the caller's stream will overwrite (second stream -> caller).
hipError_t side_stream(hipStream_t* out);
constexpr int kSlots = 8;
struct BwdEvents {
  hipEvent_t fork = nullptr;
  hipEvent_t done[kSlots] = {};
  int dev = -1;
  hipError_t create();
};
hipError_t take_events(BwdEvents** out);
void give_events(BwdEvents* e);
// Sustained bf16 MFMA rate of the current device (TFLOP/s), timed on st (synchronises on it).
hipError_t probe_mfma_rate(float* sink, double* tflops, hipStream_t st);

hipError_t launch_gather(int elt, int B, int L, int K, int D, const void* x, const int32_t* idx, void* h0, int shared,
                         hipStream_t st);
hipError_t launch_gather_rows_f32(int dtype, int B, int L, int K, int D, const void* x, const int32_t* idx,
                                  float* y32, void* ycopy, int shared, hipStream_t st);
hipError_t launch_scatter_f32_delta(int dtype, int B, int L, int K, int D, void* x, const float* h32,
                                    const int32_t* idx, int shared, hipStream_t st);
hipError_t launch_scatter_delta(int dtype, int B, int L, int K, int D, void* x, const void* h, const void* h0,
                                const int32_t* idx, int shared, hipStream_t st);

hipError_t launch_ln_fwd(int dtype, const float* x, const void* gamma, const void* beta, const float* mod, int mod_off,
                         int M, int S, int D, float eps, void* y, float* mean, float* rstd, hipStream_t st);
// ln_fwd on the routed rows x[b, idx[b, s]] of the token sequence xsrc [B, L, D] (storage type),
// also writing their fp32 values to xcopy [B*S, D].
hipError_t launch_ln_fwd_gather(int dtype, const void* xsrc, const int32_t* idx, int L, int shared, float* xcopy,
                                const void* gamma, const void* beta, const float* mod, int mod_off, int M, int S,
                                int D, float eps, void* y, float* mean, float* rstd, hipStream_t st);
// The LayerNorm output from the forward's saved statistics, bit for bit the ln_fwd result.
hipError_t launch_ln_apply(int dtype, const float* x, const void* gamma, const void* beta, const float* mod,
                           int mod_off, int M, int S, int D, const float* mean, const float* rstd, void* y,
                           hipStream_t st);
// gz = GELU(z) of the stored FC1 pre-activation (n elements, a multiple of 8), bit for bit the
// FC1 epilogue's second output.
hipError_t launch_gelu(int dtype, const void* z, void* gz, size_t n, hipStream_t st);
int ln_bwd_chunks(int S);
hipError_t launch_ln_bwd(int dtype, const float* du, const float* x, const float* mean, const float* rstd,
                         const void* gamma, const float* mod, int mod_off, const float* dres, int B, int S, int D,
                         float* dx, void* dx_act, float* part, hipStream_t st);
int colsum_chunks(int S);
hipError_t launch_colsum(int xt, const void* X, int yt, const void* Y, const float* w, int wstride, int B, int S,
                         int N, float* part, hipStream_t st);
hipError_t launch_convert(int ti, const void* x, int to, void* y, size_t n, const float* w, int wstride, int S, int D,
                          float* y32, hipStream_t st);
hipError_t launch_reduce_cols(const float* part, int R, int G, int sum_groups, int width, int half, float* out_lo,
                              float* out_hi, int out_stride, hipStream_t st, int accumulate = 0);
// Matrix-vector products of the adaLN conditioning (few rows B, bandwidth-bound in the weight):
//  rows: y[b*ldy + j] = bias[j] + sum_d x[b*ldx + d] W[j*Dd + d]   (x, W, bias storage type)
//  cols: y[b*ldy + n] (+)= sum_j x[b*ldx + j] W[j*N + n]           (x fp32, W storage type),
//        through partial sums over row chunks (scratch of gemv_cols_scratch floats).
hipError_t launch_gemv_rows(int dtype, const void* x, int ldx, const void* W, const void* bias, int B, int J, int Dd,
                            float* y, int ldy, hipStream_t st);
size_t gemv_cols_scratch(int B, int J, int N);
hipError_t launch_gemv_cols(int dtype, const float* x, int ldx, const void* W, int B, int J, int N, float* y,
                            int accumulate, float* part, hipStream_t st);
hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t st);
hipError_t launch_attn_delta(int dtype, const void* dO, const void* O, int B, int S, int H, int hd, float* delta,
                             hipStream_t st);

hipError_t launch_gemm(const GemmDesc& g, int epi, const EpiArgs& ep, hipStream_t st);
// Weight gradient dW[M x N] = sum_k A(m, k) B(n, k) over tokens k (both operands token-major)
// and db[m] = sum_k A(m, k) (optional).  part / dbpart: scratch of the sizes below.
// A weight gradient's reduction of its split-K planes (part: splits planes of n) into out and of
// its bias-gradient partial rows (dbparts rows of nb) into dbout, in part order.
struct ReduceJob {
  const float* part = nullptr;
  int splits = 1;
  size_t n = 0;
  float* out = nullptr;
  const float* dbpart = nullptr;
  int dbparts = 1;
  int nb = 0;
  float* dbout = nullptr;
  // column-sum mode (rows > 0; the LayerNorm parameter gradients): part holds rows x width
  // partials (row stride width), summed per column in the order of reduce_cols_kernel; columns
  // below half go to out, the others to dbout (either may be NULL)
  int rows = 0;
  int width = 0;
  int half = 0;
};
constexpr int kMaxReduceJobs = 6;
// With defer, the reduction the weight gradient needs (if any) is described there instead of
// launched; launch_reduce_jobs then runs up to kMaxReduceJobs of them in one launch, with the
// arithmetic and order of the single ones.
hipError_t launch_weight_grad(const GemmDesc& g, float* dw, float* db, float* part, float* dbpart, hipStream_t st,
                              ReduceJob* defer = nullptr);
hipError_t launch_reduce_jobs(const ReduceJob* jobs, int njobs, hipStream_t st);
void weight_grad_scratch(int M, int N, int K, size_t* part_floats, size_t* dbpart_floats);

bool attn_uses_mfma(int dtype, int hd);
hipError_t launch_attn_fwd(int dtype, const void* qkv, void* O, float* lse, int B, int S, int H, int D,
                           hipStream_t st);
hipError_t launch_attn_colsum(int dtype, const void* qkv, const float* lse, float* colsum, int B, int S, int H, int D,
                              hipStream_t st);
// bf16 operands as their 16-bit patterns
hipError_t launch_attn_fwd_mfma(const uint16_t* q, int ldq, const uint16_t* kv, int ldkv, uint32_t kv_elems, uint16_t* O,
                                float* lse, int B, int Sq, int Skv, int H, int D, hipStream_t st);
hipError_t launch_attn_dkv_mfma(const uint16_t* q, int ldq, uint32_t q_elems, const uint16_t* kv, int ldkv,
                                const uint16_t* dO, const float* lse, const float* delta, uint16_t* dk_out, int ldo, int B,
                                int Sq, int Skv, int H, int D, hipStream_t st);
hipError_t launch_attn_dq_mfma(const uint16_t* q, int ldq, const uint16_t* kv, int ldkv, uint32_t kv_elems,
                               const uint16_t* dO, const float* lse, const float* delta, uint16_t* dq_out, int ldo, int B,
                               int Sq, int Skv, int H, int D, hipStream_t st);
hipError_t launch_xattn_fwd(int dtype, const void* q, const void* kv, void* O, float* lse, int B, int Sq, int Skv,
                            int H, int D, hipStream_t st);
hipError_t launch_xattn_bwd(int dtype, const void* q, const void* kv, const void* O, const void* dO, const float* lse,
                            float* delta, void* dq, void* dkv, int B, int Sq, int Skv, int H, int D, hipStream_t st);
hipError_t launch_attn_bwd(int dtype, const void* qkv, const void* dO, const float* lse, const float* delta,
                           void* dqkv, int B, int S, int H, int D, hipStream_t st);

}  // namespace sr
