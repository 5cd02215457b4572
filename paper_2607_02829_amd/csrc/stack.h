// Host-side orchestration of the middle-block stack: workspace layout and the
// per-block launch sequences (forward and backward).
#pragma once
#include <string>

#include "../../include/sr.h"
#include "sr_internal.h"

namespace sr {

struct Dims {
  int B, L, D, H, F, nb, S, M;
  int dtype, kind;
  float eps;
  size_t elt;   // bytes per storage / activation element
};

struct BlockSaved {
  float *hin, *mean1, *rstd1, *lse, *h1, *mean2, *rstd2, *mod;
  void *u1, *qkv, *O, *u2, *z, *gz, *a_out, *m_out;
};

struct Scratch {
  // weight-gradient partials per kind (QKV, output projection, FC1, FC2): split planes, then room
  // for an unwanted dW; bias-gradient partial rows.  One set per kind, so that a block's four
  // reductions can run as one launch after its last weight gradient.
  float *wpart[4], *dbpart[4];
  float *g_res, *g_res2, *du, *delta, *part, *lnpart[2][2], *dmod, *gvpart;
  void *g_act[2], *dz[2], *dO, *dqkv[2], *u_rc, *gz_rc;
};

// Routing fused into the stack's boundaries: the input rows are gathered from x by idx
// (forward: x0; backward: the gradient g of x'), and the output goes back into x by the
// residual-delta scatter (forward: x' = x0 + Scatter(h - h0); backward: g + Scatter(dh - g[I])).
struct Route {
  const int32_t* idx = nullptr;   // [B or 1, S], duplicate-free rows
  void* x = nullptr;              // [B, L, D] storage type, updated in place
  int shared = 0;
};

// Carve `base` (may be null: sizes only).  Returns the bytes used.
size_t layout_saved(const Dims& d, char* base, BlockSaved* out /* [nb] or null */);
size_t layout_scratch(const Dims& d, char* base, Scratch* out /* or null */);

// With `rt`, h_in / h_out (forward) and dh_out / dh_in (backward) are unused.
hipError_t stack_fwd(const Dims& d, const sr_block_params* p, const void* cond, const void* h_in, void* h_out,
                     char* saved, hipStream_t st, const Route* rt = nullptr);
hipError_t stack_bwd(const Dims& d, const sr_block_params* p, const void* cond, const char* saved,
                     const void* dh_out, void* dh_in, const sr_block_grads* g, float* dcond, char* scratch,
                     hipStream_t st, const Route* rt = nullptr);

}  // namespace sr
