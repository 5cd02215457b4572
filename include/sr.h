/*
 * sr.h -- C ABI of libsr, the MI355X (gfx950) hot path of Sparse-Reslim:
 * random (or top-k) token selection, gather, the n2 middle transformer blocks
 * run on the routed tokens only (forward and backward), and the residual-delta
 * scatter back into the full token sequence, plus the dense keep=100% mode.
 *
 * The operations follow the paper's statement of the method:
 *   selection            Sec. 3.2 "Random token selection"; Alg. 1 stage 2; App. A.4
 *   gather / scatter     Sec. 3.2 "Residual delta formulation", Eq. (scatter)
 *   middle stack         Eq. (sparse_forward); block of Sec. 3.3
 *   dense mode           Sec. 3.4 "Architecture-agnostic design" (r = 1)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensor arguments are DEVICE pointers owned by the caller, contiguous,
 *    row-major, 16-byte aligned.  The library allocates no device memory:
 *    saved activations and scratch space are caller buffers sized by
 *    sr_workspace_bytes / sr_select_scratch_bytes.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Calls enqueue work
 *    on it and return without waiting.  The blocks backward also uses one extra
 *    stream per device (created on the first call, default priority, kept until the
 *    process ends) for its weight gradients, joined to `stream` through events: all of
 *    the call's work is complete when later work on `stream` starts.
 *  - Calls can be captured into a HIP graph (after one eager call has created the second
 *    stream and its events): they record no memset and no host synchronisation, and the
 *    backward forks and joins its second stream through events on `stream`.  A replay
 *    repeats the captured scalar arguments (seed, step, sizes).
 *  - Arguments are validated on the host before anything is enqueued; on error
 *    nothing is launched, a non-zero sr_status is returned and sr_last_error()
 *    (thread-local) describes it.  SR_EHIP reports a failed launch.
 *  - Storage dtype (sr_config.dtype): SR_F32 or SR_BF16.  Activations, weights,
 *    biases, LayerNorm parameters and the conditioning vector are stored in it;
 *    all accumulation is fp32; weight gradients and dcond are always fp32.
 *  - Non-finite values: a NaN or Inf in a sample's inputs (tokens, conditioning) or in the
 *    parameters gives non-finite values in that sample's outputs and gradients (attention mixes
 *    every token of a sample, so all of its routed rows may be affected; which elements is not
 *    specified) and in the parameter gradients; other samples' results are unchanged and rows
 *    the scatter does not touch keep their values.  Nothing is clamped or checked on the GPU.
 *  - Debugging: with SR_DEBUG=1 in the environment (read at every call), sr_gather,
 *    sr_scatter_delta and sr_routed_blocks_fwd/bwd copy idx to the host, synchronising
 *    `stream`, and return SR_EINVAL before any launch if a row is not strictly increasing
 *    inside [0, L).  Off by default (no host synchronisation on the hot path); not for use
 *    under graph capture.
 *  - Shapes: B samples, L tokens per sample, D channels, H heads (D % H == 0),
 *    F MLP width, n_blocks middle blocks; S = K (routed) or L (dense) tokens per
 *    sample inside the stack.
 *  - Support: D % 64 == 0, F % 64 == 0, D <= 2048, head dim D/H in {32, 64, 128}
 *    (bf16 with head dim 64 or 128 runs the MFMA attention kernels, fp32 storage and
 *    head dim 32 a generic fp32-accumulating kernel); 1 <= K <= L; B*L*D*elt < 2^31 bytes per
 *    token tensor, and for the block-stack calls also B*S*max(F, 3D)*4 < 2^31 with S the
 *    call's rows per sample (the S or K routed tokens; L for the dense calls), which size the
 *    internal fp32 buffers.  Anything else returns SR_EUNSUPPORTED.
 */
#ifndef SR_H
#define SR_H

#include <stddef.h>
#include <stdint.h>

#ifndef SR_API
#define SR_API __attribute__((visibility("default")))
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SR_OK = 0,
  SR_EINVAL = 1,        /* null pointer, negative size, bad enum value        */
  SR_ESHAPE = 2,        /* inconsistent shapes (K > L, D % H != 0, ...)        */
  SR_EDTYPE = 3,        /* unknown storage dtype                              */
  SR_EALIGN = 4,        /* a tensor pointer is not 16-byte aligned            */
  SR_EWORKSPACE = 5,    /* saved / scratch buffer smaller than required       */
  SR_EUNSUPPORTED = 6,  /* valid but not supported by this library            */
  SR_EHIP = 7           /* a HIP launch failed; sr_last_error() has the text  */
} sr_status;

typedef enum { SR_F32 = 0, SR_BF16 = 1 } sr_dtype;

/* Block kinds.
 * SR_BLOCK_PRELN: h1 = h + Attn(LN1(h)); h' = h1 + MLP(LN2(h1))  (Sec. 3.3).
 * SR_BLOCK_ADALN: (shift1,scale1,gate1,shift2,scale2,gate2) = c W_ada^T + b_ada per
 *   sample; h1 = h + gate1*Attn(LN0(h)*(1+scale1)+shift1);
 *   h' = h1 + gate2*MLP(LN0(h1)*(1+scale2)+shift2), LN0 = LayerNorm without affine
 *   (FiLM scale/shift and a gate from a global conditioning vector, as in the
 *   paper's EDM block, Sec. 2 "Generative forecasting"). */
typedef enum { SR_BLOCK_PRELN = 0, SR_BLOCK_ADALN = 1 } sr_block_kind;

/* Selectors.
 * SR_SEL_RANDOM: per sample, the K tokens with the smallest SplitMix64 keys
 *   key_i = mix(s_b + (i+1)*gamma), s_b = mix(s_step + (b+1)*gamma),
 *   s_step = mix(seed + (step+1)*gamma): a uniformly random K-subset
 *   (randperm(L)[:K]), ascending (Sec. 3.2; App. A.4).  A fresh `step` gives a
 *   fresh draw (Sec. 3.4 "Training and inference").
 * SR_SEL_TOPK_DIFFNORM: the K tokens with the largest
 *   score_i = sum_d (x_t[i,d] - x_prev[i,d])^2 (fp32, fixed evaluation order:
 *   16-byte chunks dealt round-robin to 64 partial sums, each summed in order,
 *   then combined by an xor butterfly 32,16,8,4,2,1; no fused multiply-add),
 *   ties to the lower index, ascending (deterministic routing ablation,
 *   App. "regularization decomposition"). */
typedef enum { SR_SEL_RANDOM = 0, SR_SEL_TOPK_DIFFNORM = 1 } sr_select_kind;

typedef struct {
  int32_t B, L, D, H, F, n_blocks;
  int32_t dtype;       /* sr_dtype */
  int32_t kind;        /* sr_block_kind */
  float ln_eps;        /* LayerNorm epsilon (the paper leaves it unstated; 1e-6 here) */
  int32_t idx_shared;  /* 1: idx is [1,K], one index set for every sample (the
                          App. A.4 listing); 0: idx is [B,K], one set per sample */
} sr_config;

/* Parameters of one block, nn.Linear layout [out, in], storage dtype, device
 * pointers.  QKV rows are ordered q, k, v; head j owns rows j*hd .. j*hd+hd-1 of
 * each.  PRELN blocks read ln*, w_qkv..b_fc2 (w_ada/b_ada may be NULL); ADALN
 * blocks read w_qkv..b_fc2 and w_ada [6D,D] / b_ada [6D] (ln* may be NULL). */
typedef struct {
  const void *ln1_w, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  const void *ln2_w, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
  const void *w_ada, *b_ada;
} sr_block_params;

/* Gradients of one block, fp32 device buffers shaped like the parameters.
 * They are OVERWRITTEN (not accumulated).  A NULL member skips that gradient;
 * members for parameters the block kind does not use are written with zeros. */
typedef struct {
  float *ln1_w, *ln1_b, *w_qkv, *b_qkv, *w_o, *b_o;
  float *ln2_w, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
  float *w_ada, *b_ada;
} sr_block_grads;

/* Text of the last error on this thread ("" if none).  The pointer stays valid
 * until the next failing call on the same thread. */
SR_API const char* sr_last_error(void);

/* Library version string. */
SR_API const char* sr_version(void);

/* Bytes of the `saved` (activations kept from forward for backward) and
 * `scratch` buffers needed by the block calls at S tokens per sample. */
SR_API sr_status sr_workspace_bytes(const sr_config* cfg, int32_t S, size_t* saved_bytes,
                             size_t* scratch_bytes);

/* Bytes of scratch sr_select_indices needs for `select_kind` (0 for random). */
SR_API sr_status sr_select_scratch_bytes(const sr_config* cfg, int32_t select_kind,
                                  size_t* scratch_bytes);

/* Token selection (Sec. 3.2; Alg. 1 stage 2; App. A.4).
 *   K: tokens kept per sample, K = floor(r*L) computed by the caller (1 <= K <= L).
 *   select_kind: sr_select_kind.  seed, step: the random draw (RANDOM only).
 *   x_t, x_prev: [B,L,D] storage dtype (TOPK only; NULL for RANDOM).
 *   idx: [B,K] int32 out (or [1,K] with idx_shared, drawn for sample 0),
 *        strictly increasing per row.
 *   scratch: sr_select_scratch_bytes bytes (may be NULL when that is 0). */
SR_API sr_status sr_select_indices(const sr_config* cfg, int32_t K, int32_t select_kind,
                            uint64_t seed, uint64_t step, const void* x_t,
                            const void* x_prev, int32_t* idx, void* scratch,
                            size_t scratch_bytes, void* stream);

/* sr_select_indices without a scratch argument and without allocating, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results and errors as sr_select_indices; the
 * SR_SEL_TOPK_DIFFNORM scores go to a device array that the library holds on each GPU it runs
 * on until the process ends (SR_SELECT_NOALLOC_MAX_TOKENS fp32 values, 4 MiB per GPU), looked
 * up once per GPU on the first call there.  B*L (L with idx_shared) above that limit returns
 * SR_EUNSUPPORTED before anything is enqueued.  Every call on one GPU shares its array: calls
 * that overlap on one GPU (different streams, threads) race and must be ordered by the caller.
 * SR_SEL_RANDOM uses no scratch and runs as in sr_select_indices. */
#define SR_SELECT_NOALLOC_MAX_TOKENS (1 << 20)
SR_API sr_status sr_select_indices_noalloc(const sr_config* cfg, int32_t K, int32_t select_kind,
                                    uint64_t seed, uint64_t step, const void* x_t,
                                    const void* x_prev, int32_t* idx, void* stream);

/* Gather (Sec. 3.2, h0 = Gather(x, I)): h0[b,k,:] = x[b, idx[b,k], :], a bit copy.
 *   x: [B,L,D] storage dtype; idx: [B,K] (or [1,K]); h0: [B,K,D] out.
 *   idx entries must lie in [0,L) (sr_select_indices guarantees it). */
SR_API sr_status sr_gather(const sr_config* cfg, int32_t K, const void* x, const int32_t* idx,
                    void* h0, void* stream);

/* Residual-delta scatter (Eq. scatter), IN PLACE on x:
 *   x[b,i,:] <- rnd( f32(x[b,i,:]) + (f32(h[b,k,:]) - f32(h0[b,k,:])) ), i = idx[b,k],
 * fp32 subtract then add, one round-to-nearest-even to the storage dtype; rows not
 * in idx are not touched (they keep x0 bit for bit).  h0 == NULL re-reads x[idx]
 * (equal to h0 by definition).  idx rows must be duplicate-free.
 * The backward of the routed step uses the same call:
 *   gather(g) -> blocks_bwd -> scatter_delta(g, dh_in, NULL, idx). */
SR_API sr_status sr_scatter_delta(const sr_config* cfg, int32_t K, void* x, const void* h,
                           const void* h0, const int32_t* idx, void* stream);

/* The n_blocks middle blocks on S tokens per sample (Eq. sparse_forward).
 *   params: host array of n_blocks sr_block_params.
 *   cond: [B,D] storage dtype (ADALN) or NULL.
 *   h_in: [B,S,D] in; h_out: [B,S,D] out (may not alias h_in).
 *   saved: activations for sr_sparse_blocks_bwd; must outlive it.
 * Inside the stack the residual stream is fp32; h_out is rounded once. */
SR_API sr_status sr_sparse_blocks_fwd(const sr_config* cfg, int32_t S,
                               const sr_block_params* params, const void* cond,
                               const void* h_in, void* h_out, void* saved,
                               size_t saved_bytes, void* scratch, size_t scratch_bytes,
                               void* stream);

/* Vector-Jacobian product of sr_sparse_blocks_fwd (same cfg, S, params, cond, saved).
 *   dh_out: [B,S,D] storage dtype in;  dh_in: [B,S,D] out (may alias dh_out).
 *   grads: host array of n_blocks sr_block_grads (fp32, overwritten).
 *   dcond: [B,D] fp32 out (ADALN; summed over blocks) or NULL. */
SR_API sr_status sr_sparse_blocks_bwd(const sr_config* cfg, int32_t S,
                               const sr_block_params* params, const void* cond,
                               const void* saved, size_t saved_bytes, const void* dh_out,
                               void* dh_in, const sr_block_grads* grads, float* dcond,
                               void* scratch, size_t scratch_bytes, void* stream);

/* Dense keep=100% mode (Sec. 3.4, r = 1): the same blocks on all L tokens. */
SR_API sr_status sr_dense_blocks_fwd(const sr_config* cfg, const sr_block_params* params,
                              const void* cond, const void* x_in, void* x_out, void* saved,
                              size_t saved_bytes, void* scratch, size_t scratch_bytes,
                              void* stream);
SR_API sr_status sr_dense_blocks_bwd(const sr_config* cfg, const sr_block_params* params,
                              const void* cond, const void* saved, size_t saved_bytes,
                              const void* dx_out, void* dx_in, const sr_block_grads* grads,
                              float* dcond, void* scratch, size_t scratch_bytes, void* stream);

/* The routed step's forward in one call (Alg. 1 stage 2): gather, the n_blocks blocks on
 * the K routed tokens, residual-delta scatter, with the gather fused into the stack's input
 * step and the scatter into the last block's output epilogue.  In place on x:
 *   x[b,i,:] <- rnd( f32(x0[b,i,:]) + (f32(h[b,k,:]) - f32(x0[b,i,:])) ),  i = idx[b,k],
 * h = the stack's output on h0 = x0[idx] rounded to the storage type; bit for bit the
 * result of sr_gather + sr_sparse_blocks_fwd + sr_scatter_delta.  Rows not in idx keep x0.
 *   idx: [B,K] (or [1,K] with idx_shared), duplicate-free rows inside [0,L).
 *   saved: sr_workspace_bytes(cfg, K) bytes; it holds what sr_routed_blocks_bwd (or
 *          sr_sparse_blocks_bwd with S = K) needs.  No scratch. */
SR_API sr_status sr_routed_blocks_fwd(const sr_config* cfg, int32_t K, const int32_t* idx,
                               const sr_block_params* params, const void* cond, void* x,
                               void* saved, size_t saved_bytes, void* stream);

/* Its backward in one call, in place on g (in: gradient of x', out: gradient of x0):
 *   g <- g + Scatter(J^T g[I] - g[I], I)  (the gradient delta rounded once, as in
 * sr_scatter_delta(g, dh_in, NULL, idx)); bit for bit the result of sr_gather(g) +
 * sr_sparse_blocks_bwd + sr_scatter_delta.  grads, dcond, scratch as for
 * sr_sparse_blocks_bwd with S = K. */
SR_API sr_status sr_routed_blocks_bwd(const sr_config* cfg, int32_t K, const int32_t* idx,
                               const sr_block_params* params, const void* cond,
                               const void* saved, size_t saved_bytes, void* g,
                               const sr_block_grads* grads, float* dcond, void* scratch,
                               size_t scratch_bytes, void* stream);

/* Asymmetric attention of the generative block's sparse middle stage (Sec. 3.4,
 * "Integration with Generative Forecasting"): queries from Sq tokens (the routed ones),
 * keys and values from Skv tokens (the whole conditioning sequence); per sample and head
 *   O = softmax(q k^T / sqrt(hd)) v   over the Skv keys,   cost O(Sq Skv D).
 * Only cfg's B, D, H and dtype are read and validated (D % 64 == 0, head dim D/H in
 * {32, 64, 128}); L, F, n_blocks, kind, ln_eps and idx_shared are ignored.
 *   q: [B,Sq,D]; kv: [B,Skv,2D] (k of head h at columns h*hd .., v at D + h*hd ..);
 *   O: [B,Sq,D] out; lse: [B,H,Sq] fp32 out, the base-2 log-sum-exp of the scaled scores.
 * bf16 with head dim 64 or 128 runs the MFMA attention kernels (the self-attention kernels,
 * given the two buffers and token counts); other cases generic kernels.  Deterministic. */
SR_API sr_status sr_cross_attention_fwd(const sr_config* cfg, int32_t Sq, int32_t Skv, const void* q,
                                 const void* kv, void* O, float* lse, void* stream);

/* Its backward: dq [B,Sq,D] and dkv [B,Skv,2D] (dk, dv in kv's layout) out, from the
 * forward's q, kv, O, lse and the output gradient dO [B,Sq,D]; delta: [B,H,Sq] fp32
 * caller scratch (receives rowsum(dO * O) per head). */
SR_API sr_status sr_cross_attention_bwd(const sr_config* cfg, int32_t Sq, int32_t Skv, const void* q,
                                 const void* kv, const void* O, const void* dO,
                                 const float* lse, void* dq, void* dkv, float* delta,
                                 void* stream);

/* The generative model's block (Sec. 3.4 "Integration with Generative Forecasting", Alg. 2
 * stage 2; App. A.1 EDM table: FiLM -> self-attention -> sigma-gated cross-attention -> MLP),
 * on S tokens per sample (the K routed ones in the sparse stage, S = L for the dense block)
 * with cross-attention to all L conditioning tokens (the asymmetric design):
 *   (shift, scale) = e W_film^T + b_film;   g = sigmoid(e W_g^T + b_g)       (per sample)
 *   u  = LN0(h) (1 + scale) + shift            LN0: LayerNorm without affine parameters
 *   h1 = h + SelfAttn(u)                       w_qkv [3D,D], b_qkv, w_o [D,D], b_o (over S tokens)
 *   h2 = h1 + g * (CrossAttn(LNc(h1), Z_c) W_oc^T + b_oc)
 *        queries LNc(h1) W_q^T + b_q (S tokens), [keys values] = Z_c W_kv^T + b_kv (L tokens,
 *        rows of w_kv [2D,D] ordered k, v, head-major within each)
 *   h' = h2 + GELU(LN2(h2) W_fc1^T + b_fc1) W_fc2^T + b_fc2
 * e: the noise embedding [B,D]; Z_c: the conditioning tokens [B,L,D]; both storage dtype and
 * shared by every block.  nn.Linear layout [out, in], storage dtype. */
typedef struct {
  const void *w_film, *b_film, *w_qkv, *b_qkv, *w_o, *b_o;
  const void *lnc_w, *lnc_b, *w_q, *b_q, *w_kv, *b_kv, *w_oc, *b_oc, *w_g, *b_g;
  const void *ln2_w, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} sr_edm_block_params;

/* Its gradients, fp32, shaped like the parameters, OVERWRITTEN; a NULL member skips one. */
typedef struct {
  float *w_film, *b_film, *w_qkv, *b_qkv, *w_o, *b_o;
  float *lnc_w, *lnc_b, *w_q, *b_q, *w_kv, *b_kv, *w_oc, *b_oc, *w_g, *b_g;
  float *ln2_w, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} sr_edm_block_grads;

/* Bytes of `saved` and `scratch` for the generative blocks at S query tokens per sample and
 * cfg->L conditioning tokens (cfg->kind and cfg->idx_shared are not used). */
SR_API sr_status sr_edm_workspace_bytes(const sr_config* cfg, int32_t S, size_t* saved_bytes,
                                 size_t* scratch_bytes);

/* cfg->n_blocks generative blocks on h_in [B,S,D] -> h_out [B,S,D] (may not alias), given the
 * noise embedding e [B,D] and the conditioning tokens zc [B,L,D] (L = cfg->L), storage dtype.
 * The residual stream is fp32 inside; h_out is rounded once.  saved: activations for
 * sr_edm_blocks_bwd (sr_edm_workspace_bytes), which must outlive it.  The sparse stage of
 * Alg. 2 is sr_gather -> this call with S = K -> sr_scatter_delta. */
SR_API sr_status sr_edm_blocks_fwd(const sr_config* cfg, int32_t S, const sr_edm_block_params* params,
                            const void* e, const void* zc, const void* h_in, void* h_out, void* saved,
                            size_t saved_bytes, void* stream);

/* Its vector-Jacobian product: dh_in [B,S,D] storage out (may alias dh_out); grads (host array
 * of n_blocks, fp32, overwritten); dzc [B,L,D] fp32 out, the gradient of the conditioning
 * tokens summed over the blocks, and de [B,D] fp32 out, that of the noise embedding summed over
 * the blocks (either may be NULL). */
SR_API sr_status sr_edm_blocks_bwd(const sr_config* cfg, int32_t S, const sr_edm_block_params* params,
                            const void* e, const void* zc, const void* saved, size_t saved_bytes,
                            const void* dh_out, void* dh_in, const sr_edm_block_grads* grads,
                            float* dzc, float* de, void* scratch, size_t scratch_bytes,
                            void* stream);

/* Debug check of an index set: *ok_dev (device int32) is set to 1 if every row of
 * idx is strictly increasing and inside [0,L), else 0. */
SR_API sr_status sr_validate_indices(const sr_config* cfg, int32_t K, const int32_t* idx,
                              int32_t* ok_dev, void* stream);

/* Attention received per token, for the attention-score selector (keep the K tokens that the
 * final block of the dense early stage attends to most: Sec. 4.4 "Random vs. learned token
 * selection", Tab. selection).  For block `block` (0-based) of the forward that
 * wrote `saved` on S tokens per sample (sr_sparse_blocks_fwd, or S = L for
 * sr_dense_blocks_fwd):
 *   colsum[b,h,j] = sum over i < S of P_h[i,j],  P_h = softmax_j(q_i . k_j / sqrt(hd)),
 * the forward's probabilities (recomputed from its saved q, k and row log-sum-exp).
 *   saved: that forward's buffer, at least sr_workspace_bytes(cfg, S) bytes, unchanged
 *          since the forward (the call only reads it).
 *   colsum: [B,H,S] fp32 out, overwritten.  Sums run in a fixed order (deterministic).
 * Per head, the S column sums add up to S up to rounding (every row of P sums to 1). */
SR_API sr_status sr_attention_colsums(const sr_config* cfg, int32_t S, const void* saved,
                               size_t saved_bytes, int32_t block, float* colsum,
                               void* stream);

/* Top-K by given scores: per sample b, score_j = sum over p < parts of planes[b,p,j],
 * added in fp32 in plane order starting from +0 (parts = H with sr_attention_colsums'
 * output gives the attention received summed over heads); the K largest scores are
 * kept, ties to the lower token index, idx ascending.
 *   planes: [B,parts,L] fp32 (or [1,parts,L] with idx_shared), finite and >= 0.
 *   idx: [B,K] int32 out (or [1,K] with idx_shared); 1 <= K <= L, parts >= 1. */
SR_API sr_status sr_select_topk_scores(const sr_config* cfg, int32_t K, const float* planes,
                                int32_t parts, int32_t* idx, void* stream);

/* Launch timing for measurement (not needed by the method).  After
 * sr_profile_start, every library launch group whose name contains `name_filter`
 * ("" or NULL = all) is timed with HIP events bound to its first and last kernel at launch
 * (hipExtLaunchKernelGGL), so a group's time is its kernels' own execution.  With no filter the
 * backward issues its weight-gradient GEMMs on the caller's stream (they normally run on
 * a second stream of the library, overlapping the rest), so each group is timed alone;
 * with a filter the overlap stays and the named groups are timed as they run.
 * sr_profile_stop waits for those events, stops recording and writes one line per
 * name: "<name> <launches> <total_ms> <algorithmic_flops> <algorithmic_bytes>\n"
 * into `out` (NUL-terminated, truncated to out_bytes); *needed receives the full
 * size.  Names: select_random, select_topk, select_topk_scores, attn_colsum, xattn_fwd,
 * xattn_bwd, gather,
 * scatter_delta, gather_f32, scatter_f32, ln_fwd, ln_bwd,
 * gemm_<op> (qkv, o, fc1, fc2, dx_fc2, dx_fc1, dx_o, dx_qkv, dw_<op>), attn_fwd,
 * attn_bwd_dkv, attn_bwd_dq, attn_bwd_delta, reduce, colsum, convert, mod. */
SR_API sr_status sr_profile_start(const char* name_filter);
SR_API sr_status sr_profile_stop(char* out, size_t out_bytes, size_t* needed);

/* Sustained bf16 matrix-core rate of the current device, for the denominator of a
 * measured roofline (not needed by the method).  Runs two launches of a register-only
 * kernel (one workgroup of eight waves per compute unit, independent 32x32x16 bf16 MFMAs,
 * no memory traffic in its loop; the first launch only lets the clock settle) on
 * `stream`, times the second with HIP events and waits for it.
 *   sink: device pointer to at least 4 writable bytes (the kernel stores one float there).
 *   tflops: host pointer; receives the achieved dense bf16 TFLOP/s (the datasheet peak is
 *   2500 at 2.4 GHz; the sustained rate reflects the clock under matrix load).
 * Errors: SR_EINVAL for a NULL argument, SR_EHIP if a launch or event call fails. */
SR_API sr_status sr_probe_mfma_rate(float* sink, double* tflops, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* SR_H */
