// C ABI of libsr (declared and documented in include/sr.h): argument validation
// on the host, then launches on the caller's stream.  Nothing is allocated here.
#include <algorithm>
#include <cstdarg>
#include <cstdlib>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/sr.h"
#include "edm.h"
#include "profile.h"
#include "stack.h"

static_assert(SR_SELECT_NOALLOC_MAX_TOKENS == sr::kSelStaticScores,
              "the header's limit is the size of the library's score array");

namespace {

thread_local std::string g_err;

sr_status fail(sr_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

sr_status hip_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return SR_OK;
  return fail(SR_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define SR_CHECK(cond, code, ...) \
  do {                            \
    if (!(cond)) return fail(code, __VA_ARGS__); \
  } while (0)

#define SR_PTR(p, name)                                                   \
  do {                                                                    \
    SR_CHECK((p) != nullptr, SR_EINVAL, "%s is NULL", name);              \
    SR_CHECK(aligned16(p), SR_EALIGN, "%s is not 16-byte aligned", name); \
  } while (0)

size_t elt_of(int dtype) { return dtype == SR_BF16 ? 2 : 4; }

// Routing-only calls (selection, gather, scatter, index validation) touch [B, L, D] tensors, whose
// byte offsets must fit 31 bits; the block stack also keeps [B*S, max(F, 3D)] fp32 buffers.
// rows: the stack's rows per sample in the call (S or K routed tokens; L when not given), which
// sizes its activation buffers.
sr_status check_cfg(const sr_config* c, bool routing_only = false, int64_t rows = 0) {
  SR_CHECK(c != nullptr, SR_EINVAL, "cfg is NULL");
  SR_CHECK(c->dtype == SR_F32 || c->dtype == SR_BF16, SR_EDTYPE, "unknown dtype %d", c->dtype);
  SR_CHECK(c->kind == SR_BLOCK_PRELN || c->kind == SR_BLOCK_ADALN, SR_EINVAL, "unknown block kind %d", c->kind);
  SR_CHECK(c->B >= 1 && c->L >= 1 && c->D >= 1 && c->H >= 1 && c->F >= 1 && c->n_blocks >= 0, SR_EINVAL,
           "sizes must be positive (B=%d L=%d D=%d H=%d F=%d n_blocks=%d)", c->B, c->L, c->D, c->H, c->F,
           c->n_blocks);
  SR_CHECK(c->D % c->H == 0, SR_ESHAPE, "D=%d is not a multiple of H=%d", c->D, c->H);
  SR_CHECK(c->D % 64 == 0 && c->F % 64 == 0, SR_EUNSUPPORTED, "D=%d and F=%d must be multiples of 64", c->D, c->F);
  SR_CHECK(c->D <= 2048, SR_EUNSUPPORTED, "D=%d > 2048", c->D);
  const int hd = c->D / c->H;
  SR_CHECK(hd == 32 || hd == 64 || hd == 128, SR_EUNSUPPORTED, "head dim %d not in {32, 64, 128}", hd);
  SR_CHECK(c->ln_eps > 0.f, SR_EINVAL, "ln_eps must be > 0");
  SR_CHECK(c->idx_shared == 0 || c->idx_shared == 1, SR_EINVAL, "idx_shared must be 0 or 1");
  const size_t tok = (size_t)c->B * c->L * c->D * (c->dtype == SR_BF16 ? 2 : 4);
  SR_CHECK(tok < (1ull << 31), SR_EUNSUPPORTED, "token tensors beyond 2 GiB are not supported");
  if (!routing_only) {
    const int64_t r = rows > 0 && rows <= c->L ? rows : c->L;
    const size_t big = (size_t)c->B * (size_t)r * (size_t)std::max(c->F, 3 * c->D) * 4;
    SR_CHECK(big < (1ull << 31), SR_EUNSUPPORTED,
             "stack buffers beyond 2 GiB are not supported (B=%d x %lld rows x max(F, 3D) x 4 bytes)", c->B,
             (long long)r);
  }
  return SR_OK;
}

// SR_DEBUG=1 in the environment (read at every call): calls that take an index set copy it to
// the host (synchronising the stream) and reject one that is not strictly increasing inside
// [0, L) before launching anything.
sr_status debug_check_indices(const sr_config* cfg, int32_t K, const int32_t* idx, hipStream_t st) {
  const char* v = getenv("SR_DEBUG");
  if (!(v && v[0] == '1')) return SR_OK;
  const int rows = cfg->idx_shared ? 1 : cfg->B;
  std::vector<int32_t> h((size_t)rows * K);
  hipError_t e = hipMemcpyAsync(h.data(), idx, h.size() * sizeof(int32_t), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_status(e, "SR_DEBUG index check");
  for (int r = 0; r < rows; ++r)
    for (int k = 0; k < K; ++k) {
      const int32_t x = h[(size_t)r * K + k];
      const bool ok = x >= 0 && x < cfg->L && (k == 0 || x > h[(size_t)r * K + k - 1]);
      SR_CHECK(ok, SR_EINVAL, "SR_DEBUG: idx[%d][%d] = %d breaks a strictly increasing index set inside [0, L=%d)",
               r, k, x, cfg->L);
    }
  return SR_OK;
}

sr::Dims dims_of(const sr_config* c, int S) {
  sr::Dims d;
  d.B = c->B; d.L = c->L; d.D = c->D; d.H = c->H; d.F = c->F; d.nb = c->n_blocks;
  d.S = S; d.M = c->B * S;
  d.dtype = c->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  d.kind = c->kind;
  d.eps = c->ln_eps;
  d.elt = elt_of(c->dtype);
  return d;
}

sr_status check_params(const sr_config* c, const sr_block_params* p, const void* cond) {
  SR_CHECK(p != nullptr || c->n_blocks == 0, SR_EINVAL, "params is NULL");
  for (int i = 0; i < c->n_blocks; ++i) {
    const sr_block_params& w = p[i];
    const void* common[] = {w.w_qkv, w.b_qkv, w.w_o, w.b_o, w.w_fc1, w.b_fc1, w.w_fc2, w.b_fc2};
    for (const void* q : common) {
      SR_CHECK(q != nullptr, SR_EINVAL, "block %d: a weight or bias pointer is NULL", i);
      SR_CHECK(aligned16(q), SR_EALIGN, "block %d: a weight or bias pointer is not 16-byte aligned", i);
    }
    // the row kernels read gamma / beta and the modulation weights with 8- and 16-byte loads
    if (c->kind == SR_BLOCK_PRELN) {
      const void* ln[] = {w.ln1_w, w.ln1_b, w.ln2_w, w.ln2_b};
      for (const void* q : ln) {
        SR_CHECK(q != nullptr, SR_EINVAL, "block %d: a LayerNorm parameter is NULL", i);
        SR_CHECK(aligned16(q), SR_EALIGN, "block %d: a LayerNorm parameter is not 16-byte aligned", i);
      }
    } else {
      SR_CHECK(w.w_ada && w.b_ada, SR_EINVAL, "block %d: adaLN needs w_ada and b_ada", i);
      SR_CHECK(aligned16(w.w_ada) && aligned16(w.b_ada), SR_EALIGN,
               "block %d: w_ada or b_ada is not 16-byte aligned", i);
    }
  }
  if (c->kind == SR_BLOCK_ADALN) SR_PTR(cond, "cond");
  return SR_OK;
}

sr_status check_ws(const sr_config* c, int S, const void* saved, size_t saved_bytes, const void* scratch,
                   size_t scratch_bytes, bool need_scratch) {
  size_t sb = 0, cb = 0;
  sr_status s = sr_workspace_bytes(c, S, &sb, &cb);
  if (s != SR_OK) return s;
  SR_PTR(saved, "saved");
  SR_CHECK(saved_bytes >= sb, SR_EWORKSPACE, "saved buffer has %zu bytes, needs %zu", saved_bytes, sb);
  if (need_scratch) {
    SR_PTR(scratch, "scratch");
    SR_CHECK(scratch_bytes >= cb, SR_EWORKSPACE, "scratch buffer has %zu bytes, needs %zu", scratch_bytes, cb);
  }
  return SR_OK;
}

}  // namespace

extern "C" {

const char* sr_last_error(void) { return g_err.c_str(); }

const char* sr_version(void) { return "libsr 0.1 (gfx950)"; }

sr_status sr_workspace_bytes(const sr_config* cfg, int32_t S, size_t* saved_bytes, size_t* scratch_bytes) {
  sr_status s = check_cfg(cfg, false, S);
  if (s != SR_OK) return s;
  SR_CHECK(S >= 1, SR_EINVAL, "S=%d must be >= 1", S);
  sr::Dims d = dims_of(cfg, S);
  if (saved_bytes) *saved_bytes = sr::layout_saved(d, nullptr, nullptr);
  if (scratch_bytes) *scratch_bytes = sr::layout_scratch(d, nullptr, nullptr);
  return SR_OK;
}

sr_status sr_select_scratch_bytes(const sr_config* cfg, int32_t select_kind, size_t* scratch_bytes) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(scratch_bytes != nullptr, SR_EINVAL, "scratch_bytes is NULL");
  SR_CHECK(select_kind == SR_SEL_RANDOM || select_kind == SR_SEL_TOPK_DIFFNORM, SR_EINVAL, "unknown selector %d",
           select_kind);
  *scratch_bytes = select_kind == SR_SEL_RANDOM ? 0 : (size_t)cfg->B * cfg->L * 4;
  return SR_OK;
}

sr_status sr_select_indices(const sr_config* cfg, int32_t K, int32_t select_kind, uint64_t seed, uint64_t step,
                            const void* x_t, const void* x_prev, int32_t* idx, void* scratch, size_t scratch_bytes,
                            void* stream) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_PTR(idx, "idx");
  const int rows = cfg->idx_shared ? 1 : cfg->B;
  hipStream_t st = (hipStream_t)stream;
  if (select_kind == SR_SEL_RANDOM) {
    sr::ProfScope ps("select_random", 0, (double)rows * K * 4, st);
    return hip_status(sr::launch_select_random(rows, cfg->L, K, seed, step, idx, st), "select_random");
  }
  SR_CHECK(select_kind == SR_SEL_TOPK_DIFFNORM, SR_EINVAL, "unknown selector %d", select_kind);
  SR_PTR(x_t, "x_t");
  SR_PTR(x_prev, "x_prev");
  SR_PTR(scratch, "scratch");
  SR_CHECK(scratch_bytes >= (size_t)cfg->B * cfg->L * 4, SR_EWORKSPACE, "top-k scratch needs %zu bytes",
           (size_t)cfg->B * cfg->L * 4);
  const int dt = cfg->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  sr::ProfScope ps("select_topk", 0, (double)rows * cfg->L * cfg->D * 2 * elt_of(cfg->dtype), st);
  return hip_status(sr::launch_select_topk(dt, rows, cfg->L, cfg->D, K, x_t, x_prev, (float*)scratch, idx, st),
                    "select_topk");
}

sr_status sr_select_indices_noalloc(const sr_config* cfg, int32_t K, int32_t select_kind, uint64_t seed,
                                    uint64_t step, const void* x_t, const void* x_prev, int32_t* idx,
                                    void* stream) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_PTR(idx, "idx");
  const int rows = cfg->idx_shared ? 1 : cfg->B;
  hipStream_t st = (hipStream_t)stream;
  if (select_kind == SR_SEL_RANDOM) {   // needs no scratch: the same launch as sr_select_indices
    sr::ProfScope ps("select_random", 0, (double)rows * K * 4, st);
    return hip_status(sr::launch_select_random(rows, cfg->L, K, seed, step, idx, st), "select_random");
  }
  SR_CHECK(select_kind == SR_SEL_TOPK_DIFFNORM, SR_EINVAL, "unknown selector %d", select_kind);
  SR_PTR(x_t, "x_t");
  SR_PTR(x_prev, "x_prev");
  SR_CHECK((size_t)rows * cfg->L <= (size_t)SR_SELECT_NOALLOC_MAX_TOKENS, SR_EUNSUPPORTED,
           "top-k selection without allocation scores at most %d tokens per call (B*L = %zu)",
           SR_SELECT_NOALLOC_MAX_TOKENS, (size_t)rows * cfg->L);
  float* score = nullptr;
  if ((s = hip_status(sr::select_static_scratch(&score), "select_static_scratch")) != SR_OK) return s;
  const int dt = cfg->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  sr::ProfScope ps("select_topk", 0, (double)rows * cfg->L * cfg->D * 2 * elt_of(cfg->dtype), st);
  return hip_status(sr::launch_select_topk(dt, rows, cfg->L, cfg->D, K, x_t, x_prev, score, idx, st),
                    "select_topk");
}

sr_status sr_gather(const sr_config* cfg, int32_t K, const void* x, const int32_t* idx, void* h0, void* stream) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_PTR(x, "x");
  SR_PTR(idx, "idx");
  SR_PTR(h0, "h0");
  if ((s = debug_check_indices(cfg, K, idx, (hipStream_t)stream)) != SR_OK) return s;
  sr::ProfScope ps("gather", 0, 2.0 * cfg->B * K * cfg->D * elt_of(cfg->dtype) + 4.0 * cfg->B * K, (hipStream_t)stream);
  return hip_status(sr::launch_gather((int)elt_of(cfg->dtype), cfg->B, cfg->L, K, cfg->D, x, idx, h0,
                                      cfg->idx_shared, (hipStream_t)stream),
                    "gather");
}

sr_status sr_scatter_delta(const sr_config* cfg, int32_t K, void* x, const void* h, const void* h0,
                           const int32_t* idx, void* stream) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_PTR(x, "x");
  SR_PTR(h, "h");
  SR_PTR(idx, "idx");
  if (h0) SR_CHECK(aligned16(h0), SR_EALIGN, "h0 is not 16-byte aligned");
  if ((s = debug_check_indices(cfg, K, idx, (hipStream_t)stream)) != SR_OK) return s;
  const int dt = cfg->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  sr::ProfScope ps("scatter_delta", 0, (h0 ? 4.0 : 3.0) * cfg->B * K * cfg->D * elt_of(cfg->dtype) + 4.0 * cfg->B * K,
                   (hipStream_t)stream);
  return hip_status(sr::launch_scatter_delta(dt, cfg->B, cfg->L, K, cfg->D, x, h, h0, idx, cfg->idx_shared,
                                             (hipStream_t)stream),
                    "scatter_delta");
}

sr_status sr_sparse_blocks_fwd(const sr_config* cfg, int32_t S, const sr_block_params* params, const void* cond,
                               const void* h_in, void* h_out, void* saved, size_t saved_bytes, void* scratch,
                               size_t scratch_bytes, void* stream) {
  (void)scratch; (void)scratch_bytes;
  sr_status s = check_cfg(cfg, false, S);
  if (s != SR_OK) return s;
  SR_CHECK(S >= 1 && S <= cfg->L, SR_ESHAPE, "S=%d outside [1, L=%d]", S, cfg->L);
  SR_CHECK(cfg->n_blocks >= 1, SR_EINVAL, "n_blocks must be >= 1");
  if ((s = check_params(cfg, params, cond)) != SR_OK) return s;
  SR_PTR(h_in, "h_in");
  SR_PTR(h_out, "h_out");
  SR_CHECK(h_in != h_out, SR_EINVAL, "h_out may not alias h_in");
  if ((s = check_ws(cfg, S, saved, saved_bytes, scratch, scratch_bytes, false)) != SR_OK) return s;
  sr::Dims d = dims_of(cfg, S);
  return hip_status(sr::stack_fwd(d, params, cond, h_in, h_out, (char*)saved, (hipStream_t)stream), "blocks_fwd");
}

sr_status sr_sparse_blocks_bwd(const sr_config* cfg, int32_t S, const sr_block_params* params, const void* cond,
                               const void* saved, size_t saved_bytes, const void* dh_out, void* dh_in,
                               const sr_block_grads* grads, float* dcond, void* scratch, size_t scratch_bytes,
                               void* stream) {
  sr_status s = check_cfg(cfg, false, S);
  if (s != SR_OK) return s;
  SR_CHECK(S >= 1 && S <= cfg->L, SR_ESHAPE, "S=%d outside [1, L=%d]", S, cfg->L);
  SR_CHECK(cfg->n_blocks >= 1, SR_EINVAL, "n_blocks must be >= 1");
  if ((s = check_params(cfg, params, cond)) != SR_OK) return s;
  SR_PTR(dh_out, "dh_out");
  SR_PTR(dh_in, "dh_in");
  SR_CHECK(grads != nullptr, SR_EINVAL, "grads is NULL");
  if (dcond) SR_CHECK(aligned16(dcond), SR_EALIGN, "dcond is not 16-byte aligned");
  if ((s = check_ws(cfg, S, saved, saved_bytes, scratch, scratch_bytes, true)) != SR_OK) return s;
  sr::Dims d = dims_of(cfg, S);
  return hip_status(sr::stack_bwd(d, params, cond, (const char*)saved, dh_out, dh_in, grads,
                                  cfg->kind == SR_BLOCK_ADALN ? dcond : nullptr, (char*)scratch, (hipStream_t)stream),
                    "blocks_bwd");
}

sr_status sr_routed_blocks_fwd(const sr_config* cfg, int32_t K, const int32_t* idx, const sr_block_params* params,
                               const void* cond, void* x, void* saved, size_t saved_bytes, void* stream) {
  sr_status s = check_cfg(cfg, false, K);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_CHECK(cfg->n_blocks >= 1, SR_EINVAL, "n_blocks must be >= 1");
  if ((s = check_params(cfg, params, cond)) != SR_OK) return s;
  SR_PTR(idx, "idx");
  SR_PTR(x, "x");
  if ((s = check_ws(cfg, K, saved, saved_bytes, nullptr, 0, false)) != SR_OK) return s;
  if ((s = debug_check_indices(cfg, K, idx, (hipStream_t)stream)) != SR_OK) return s;
  sr::Dims d = dims_of(cfg, K);
  sr::Route rt;
  rt.idx = idx; rt.x = x; rt.shared = cfg->idx_shared;
  return hip_status(sr::stack_fwd(d, params, cond, nullptr, nullptr, (char*)saved, (hipStream_t)stream, &rt),
                    "routed_blocks_fwd");
}

sr_status sr_routed_blocks_bwd(const sr_config* cfg, int32_t K, const int32_t* idx, const sr_block_params* params,
                               const void* cond, const void* saved, size_t saved_bytes, void* g,
                               const sr_block_grads* grads, float* dcond, void* scratch, size_t scratch_bytes,
                               void* stream) {
  sr_status s = check_cfg(cfg, false, K);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_CHECK(cfg->n_blocks >= 1, SR_EINVAL, "n_blocks must be >= 1");
  if ((s = check_params(cfg, params, cond)) != SR_OK) return s;
  SR_PTR(idx, "idx");
  SR_PTR(g, "g");
  SR_CHECK(grads != nullptr, SR_EINVAL, "grads is NULL");
  if (dcond) SR_CHECK(aligned16(dcond), SR_EALIGN, "dcond is not 16-byte aligned");
  if ((s = check_ws(cfg, K, saved, saved_bytes, scratch, scratch_bytes, true)) != SR_OK) return s;
  if ((s = debug_check_indices(cfg, K, idx, (hipStream_t)stream)) != SR_OK) return s;
  sr::Dims d = dims_of(cfg, K);
  sr::Route rt;
  rt.idx = idx; rt.x = g; rt.shared = cfg->idx_shared;
  return hip_status(sr::stack_bwd(d, params, cond, (const char*)saved, nullptr, nullptr, grads,
                                  cfg->kind == SR_BLOCK_ADALN ? dcond : nullptr, (char*)scratch, (hipStream_t)stream,
                                  &rt),
                    "routed_blocks_bwd");
}

sr_status sr_dense_blocks_fwd(const sr_config* cfg, const sr_block_params* params, const void* cond,
                              const void* x_in, void* x_out, void* saved, size_t saved_bytes, void* scratch,
                              size_t scratch_bytes, void* stream) {
  sr_status s = check_cfg(cfg);
  if (s != SR_OK) return s;
  return sr_sparse_blocks_fwd(cfg, cfg->L, params, cond, x_in, x_out, saved, saved_bytes, scratch, scratch_bytes,
                              stream);
}

sr_status sr_dense_blocks_bwd(const sr_config* cfg, const sr_block_params* params, const void* cond,
                              const void* saved, size_t saved_bytes, const void* dx_out, void* dx_in,
                              const sr_block_grads* grads, float* dcond, void* scratch, size_t scratch_bytes,
                              void* stream) {
  sr_status s = check_cfg(cfg);
  if (s != SR_OK) return s;
  return sr_sparse_blocks_bwd(cfg, cfg->L, params, cond, saved, saved_bytes, dx_out, dx_in, grads, dcond, scratch,
                              scratch_bytes, stream);
}

sr_status sr_attention_colsums(const sr_config* cfg, int32_t S, const void* saved, size_t saved_bytes, int32_t block,
                               float* colsum, void* stream) {
  sr_status s = check_cfg(cfg, false, S);
  if (s != SR_OK) return s;
  SR_CHECK(S >= 1 && S <= cfg->L, SR_ESHAPE, "S=%d outside [1, L=%d]", S, cfg->L);
  SR_CHECK(block >= 0 && block < cfg->n_blocks, SR_EINVAL, "block %d outside [0, n_blocks=%d)", block,
           cfg->n_blocks);
  if ((s = check_ws(cfg, S, saved, saved_bytes, nullptr, 0, false)) != SR_OK) return s;
  SR_PTR(colsum, "colsum");
  sr::Dims d = dims_of(cfg, S);
  std::vector<sr::BlockSaved> bs((size_t)cfg->n_blocks);
  sr::layout_saved(d, (char*)saved, bs.data());
  const int hd = cfg->D / cfg->H;
  hipStream_t st = (hipStream_t)stream;
  sr::ProfScope ps("attn_colsum", 2.0 * cfg->B * cfg->H * (double)S * S * hd,
                   (double)cfg->B * S * 2 * cfg->D * elt_of(cfg->dtype) + 8.0 * cfg->B * cfg->H * S, st);
  return hip_status(sr::launch_attn_colsum(d.dtype, bs[block].qkv, bs[block].lse, colsum, cfg->B, S, cfg->H, cfg->D,
                                           st),
                    "attn_colsum");
}

sr_status sr_select_topk_scores(const sr_config* cfg, int32_t K, const float* planes, int32_t parts, int32_t* idx,
                                void* stream) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_CHECK(parts >= 1, SR_EINVAL, "parts=%d must be >= 1", parts);
  const int rows = cfg->idx_shared ? 1 : cfg->B;
  SR_CHECK((size_t)rows * parts * cfg->L * 4 < (1ull << 31), SR_EUNSUPPORTED, "score planes beyond 2 GiB");
  SR_PTR(planes, "planes");
  SR_PTR(idx, "idx");
  hipStream_t st = (hipStream_t)stream;
  sr::ProfScope ps("select_topk_scores", 0, (double)rows * parts * cfg->L * 4 + (double)rows * K * 4, st);
  return hip_status(sr::launch_select_topk_planes(rows, cfg->L, K, parts, planes, idx, st), "select_topk_scores");
}

namespace {
// The asymmetric attention reads only B, D, H and the storage type of cfg.
sr_status check_xattn(const sr_config* c, int32_t Sq, int32_t Skv) {
  SR_CHECK(c != nullptr, SR_EINVAL, "cfg is NULL");
  SR_CHECK(c->dtype == SR_F32 || c->dtype == SR_BF16, SR_EDTYPE, "unknown dtype %d", c->dtype);
  SR_CHECK(c->B >= 1 && c->D >= 1 && c->H >= 1, SR_EINVAL, "sizes must be positive (B=%d D=%d H=%d)", c->B, c->D,
           c->H);
  SR_CHECK(c->D % c->H == 0, SR_ESHAPE, "D=%d is not a multiple of H=%d", c->D, c->H);
  SR_CHECK(c->D % 64 == 0, SR_EUNSUPPORTED, "D=%d must be a multiple of 64", c->D);
  const int hd = c->D / c->H;
  SR_CHECK(hd == 32 || hd == 64 || hd == 128, SR_EUNSUPPORTED, "head dim %d not in {32, 64, 128}", hd);
  const sr_config* cfg = c;
  SR_CHECK(Sq >= 1 && Skv >= 1, SR_ESHAPE, "Sq=%d and Skv=%d must be >= 1", Sq, Skv);
  const size_t e = elt_of(cfg->dtype);
  SR_CHECK((size_t)cfg->B * Skv * 2 * cfg->D * e < (1ull << 31) && (size_t)cfg->B * Sq * cfg->D * e < (1ull << 31),
           SR_EUNSUPPORTED, "attention operands beyond 2 GiB are not supported");
  return SR_OK;
}
}  // namespace

sr_status sr_cross_attention_fwd(const sr_config* cfg, int32_t Sq, int32_t Skv, const void* q, const void* kv,
                                 void* O, float* lse, void* stream) {
  sr_status s = check_xattn(cfg, Sq, Skv);
  if (s != SR_OK) return s;
  SR_PTR(q, "q");
  SR_PTR(kv, "kv");
  SR_PTR(O, "O");
  SR_PTR(lse, "lse");
  hipStream_t st = (hipStream_t)stream;
  const int dt = cfg->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  const size_t e = elt_of(cfg->dtype);
  sr::ProfScope ps("xattn_fwd", 4.0 * cfg->B * (double)Sq * Skv * cfg->D,
                   (double)cfg->B * (2.0 * Sq + 2.0 * Skv) * cfg->D * e, st);
  return hip_status(sr::launch_xattn_fwd(dt, q, kv, O, lse, cfg->B, Sq, Skv, cfg->H, cfg->D, st), "xattn_fwd");
}

sr_status sr_cross_attention_bwd(const sr_config* cfg, int32_t Sq, int32_t Skv, const void* q, const void* kv,
                                 const void* O, const void* dO, const float* lse, void* dq, void* dkv, float* delta,
                                 void* stream) {
  sr_status s = check_xattn(cfg, Sq, Skv);
  if (s != SR_OK) return s;
  SR_PTR(q, "q");
  SR_PTR(kv, "kv");
  SR_PTR(O, "O");
  SR_PTR(dO, "dO");
  SR_PTR(lse, "lse");
  SR_PTR(dq, "dq");
  SR_PTR(dkv, "dkv");
  SR_PTR(delta, "delta");
  hipStream_t st = (hipStream_t)stream;
  const int dt = cfg->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  const size_t e = elt_of(cfg->dtype);
  sr::ProfScope ps("xattn_bwd", 8.0 * cfg->B * (double)Sq * Skv * cfg->D,
                   (double)cfg->B * (5.0 * Sq + 4.0 * Skv) * cfg->D * e, st);
  return hip_status(sr::launch_xattn_bwd(dt, q, kv, O, dO, lse, delta, dq, dkv, cfg->B, Sq, Skv, cfg->H, cfg->D, st),
                    "xattn_bwd");
}

namespace {
// The generative blocks read B, L (conditioning tokens), D, H, F, n_blocks, dtype and ln_eps.
sr_status check_edm(const sr_config* c, int32_t S) {
  SR_CHECK(c != nullptr, SR_EINVAL, "cfg is NULL");
  SR_CHECK(c->dtype == SR_F32 || c->dtype == SR_BF16, SR_EDTYPE, "unknown dtype %d", c->dtype);
  SR_CHECK(c->B >= 1 && c->L >= 1 && c->D >= 1 && c->H >= 1 && c->F >= 1 && c->n_blocks >= 1, SR_EINVAL,
           "sizes must be positive (B=%d L=%d D=%d H=%d F=%d n_blocks=%d)", c->B, c->L, c->D, c->H, c->F,
           c->n_blocks);
  SR_CHECK(S >= 1, SR_ESHAPE, "S=%d must be >= 1", S);
  SR_CHECK(c->D % c->H == 0, SR_ESHAPE, "D=%d is not a multiple of H=%d", c->D, c->H);
  SR_CHECK(c->D % 64 == 0 && c->F % 64 == 0, SR_EUNSUPPORTED, "D=%d and F=%d must be multiples of 64", c->D, c->F);
  SR_CHECK(c->D <= 2048, SR_EUNSUPPORTED, "D=%d > 2048", c->D);
  const int hd = c->D / c->H;
  SR_CHECK(hd == 32 || hd == 64 || hd == 128, SR_EUNSUPPORTED, "head dim %d not in {32, 64, 128}", hd);
  SR_CHECK(c->ln_eps > 0.f, SR_EINVAL, "ln_eps must be > 0");
  const size_t rows = (size_t)c->B * std::max<int32_t>(S, c->L);
  SR_CHECK(rows * (size_t)std::max(c->F, 3 * c->D) * 4 < (1ull << 31), SR_EUNSUPPORTED,
           "stack buffers beyond 2 GiB are not supported");
  return SR_OK;
}

sr::EdmDims edm_dims(const sr_config* c, int S) {
  sr::EdmDims d;
  d.B = c->B; d.L = c->L; d.D = c->D; d.H = c->H; d.F = c->F; d.nb = c->n_blocks; d.S = S;
  d.M = c->B * S; d.Mc = c->B * c->L;
  d.dtype = c->dtype == SR_BF16 ? sr::kBF16 : sr::kF32;
  d.eps = c->ln_eps;
  d.elt = elt_of(c->dtype);
  return d;
}

sr_status check_edm_params(const sr_config* c, const sr_edm_block_params* p) {
  SR_CHECK(p != nullptr, SR_EINVAL, "params is NULL");
  for (int i = 0; i < c->n_blocks; ++i) {
    const sr_edm_block_params& w = p[i];
    const void* all[] = {w.w_film, w.b_film, w.w_qkv, w.b_qkv, w.w_o, w.b_o, w.lnc_w, w.lnc_b, w.w_q, w.b_q, w.w_kv,
                         w.b_kv, w.w_oc, w.b_oc, w.w_g, w.b_g, w.ln2_w, w.ln2_b, w.w_fc1, w.b_fc1, w.w_fc2, w.b_fc2};
    for (const void* q : all) {
      SR_CHECK(q != nullptr, SR_EINVAL, "generative block %d: a parameter pointer is NULL", i);
      SR_CHECK(aligned16(q), SR_EALIGN, "generative block %d: a parameter pointer is not 16-byte aligned", i);
    }
  }
  return SR_OK;
}
}  // namespace

sr_status sr_edm_workspace_bytes(const sr_config* cfg, int32_t S, size_t* saved_bytes, size_t* scratch_bytes) {
  sr_status s = check_edm(cfg, S);
  if (s != SR_OK) return s;
  sr::EdmDims d = edm_dims(cfg, S);
  if (saved_bytes) *saved_bytes = sr::edm_layout_saved(d, nullptr, nullptr);
  if (scratch_bytes) *scratch_bytes = sr::edm_layout_scratch(d, nullptr, nullptr);
  return SR_OK;
}

sr_status sr_edm_blocks_fwd(const sr_config* cfg, int32_t S, const sr_edm_block_params* params, const void* e,
                            const void* zc, const void* h_in, void* h_out, void* saved, size_t saved_bytes,
                            void* stream) {
  sr_status s = check_edm(cfg, S);
  if (s != SR_OK) return s;
  if ((s = check_edm_params(cfg, params)) != SR_OK) return s;
  SR_PTR(e, "e");
  SR_PTR(zc, "zc");
  SR_PTR(h_in, "h_in");
  SR_PTR(h_out, "h_out");
  SR_CHECK(h_in != h_out, SR_EINVAL, "h_out may not alias h_in");
  size_t sb = 0;
  sr_edm_workspace_bytes(cfg, S, &sb, nullptr);
  SR_PTR(saved, "saved");
  SR_CHECK(saved_bytes >= sb, SR_EWORKSPACE, "saved buffer has %zu bytes, needs %zu", saved_bytes, sb);
  return hip_status(sr::edm_fwd(edm_dims(cfg, S), params, e, zc, h_in, h_out, (char*)saved, (hipStream_t)stream),
                    "edm_blocks_fwd");
}

sr_status sr_edm_blocks_bwd(const sr_config* cfg, int32_t S, const sr_edm_block_params* params, const void* e,
                            const void* zc, const void* saved, size_t saved_bytes, const void* dh_out, void* dh_in,
                            const sr_edm_block_grads* grads, float* dzc, float* de, void* scratch,
                            size_t scratch_bytes, void* stream) {
  sr_status s = check_edm(cfg, S);
  if (s != SR_OK) return s;
  if ((s = check_edm_params(cfg, params)) != SR_OK) return s;
  SR_PTR(e, "e");
  SR_PTR(zc, "zc");
  SR_PTR(dh_out, "dh_out");
  SR_PTR(dh_in, "dh_in");
  SR_CHECK(grads != nullptr, SR_EINVAL, "grads is NULL");
  if (dzc) SR_CHECK(aligned16(dzc), SR_EALIGN, "dzc is not 16-byte aligned");
  if (de) SR_CHECK(aligned16(de), SR_EALIGN, "de is not 16-byte aligned");
  size_t sb = 0, cb = 0;
  sr_edm_workspace_bytes(cfg, S, &sb, &cb);
  SR_PTR(saved, "saved");
  SR_CHECK(saved_bytes >= sb, SR_EWORKSPACE, "saved buffer has %zu bytes, needs %zu", saved_bytes, sb);
  SR_PTR(scratch, "scratch");
  SR_CHECK(scratch_bytes >= cb, SR_EWORKSPACE, "scratch buffer has %zu bytes, needs %zu", scratch_bytes, cb);
  return hip_status(sr::edm_bwd(edm_dims(cfg, S), params, e, zc, (const char*)saved, dh_out, dh_in, grads, dzc, de,
                                (char*)scratch, (hipStream_t)stream),
                    "edm_blocks_bwd");
}

sr_status sr_probe_mfma_rate(float* sink, double* tflops, void* stream) {
  SR_CHECK(sink != nullptr && tflops != nullptr, SR_EINVAL, "sink and tflops must not be NULL");
  return hip_status(sr::probe_mfma_rate(sink, tflops, (hipStream_t)stream), "probe_mfma_rate");
}

sr_status sr_validate_indices(const sr_config* cfg, int32_t K, const int32_t* idx, int32_t* ok_dev, void* stream) {
  sr_status s = check_cfg(cfg, true);
  if (s != SR_OK) return s;
  SR_CHECK(K >= 1 && K <= cfg->L, SR_ESHAPE, "K=%d outside [1, L=%d]", K, cfg->L);
  SR_PTR(idx, "idx");
  SR_CHECK(ok_dev != nullptr, SR_EINVAL, "ok_dev is NULL");
  const int rows = cfg->idx_shared ? 1 : cfg->B;
  return hip_status(sr::launch_validate(idx, rows, K, cfg->L, ok_dev, (hipStream_t)stream), "validate_indices");
}

}  // extern "C"
