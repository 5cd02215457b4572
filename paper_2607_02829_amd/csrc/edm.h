// Host-side orchestration of the generative model's blocks (FiLM, self-attention on the S
// routed tokens, sigma-gated cross-attention to all L conditioning tokens, MLP): workspace
// layout and the launch sequences of the forward and its vector-Jacobian product.
#pragma once
#include "../../include/sr.h"
#include "sr_internal.h"

namespace sr {

struct EdmDims {
  int B, L, D, H, F, nb, S;
  int M, Mc;      // B*S query rows, B*L conditioning rows
  int dtype;
  float eps;
  size_t elt;     // bytes per storage element
};

struct EdmSaved {
  float *mod, *hin, *mean0, *rstd0, *lse, *h1, *meanc, *rstdc, *lsec, *h2, *mean2, *rstd2;
  void *u, *qkv, *O, *uc, *qc, *kvc, *Oc, *c_out, *u2, *z, *gz;
};

struct EdmScratch {
  float *g_res, *g_res2, *du, *delta, *wpart, *dbpart, *part, *lnpart, *dmod, *gvpart;
  void *g_act, *dc, *dz, *dO, *dqkv, *dqc, *dkvc;
};

// Carve `base` (may be null: sizes only).  Returns the bytes used.
size_t edm_layout_saved(const EdmDims& d, char* base, EdmSaved* out /* [nb] or null */);
size_t edm_layout_scratch(const EdmDims& d, char* base, EdmScratch* out /* or null */);

hipError_t edm_fwd(const EdmDims& d, const sr_edm_block_params* p, const void* e_sig, const void* zc,
                   const void* h_in, void* h_out, char* saved, hipStream_t st);
hipError_t edm_bwd(const EdmDims& d, const sr_edm_block_params* p, const void* e_sig, const void* zc,
                   const char* saved, const void* dh_out, void* dh_in, const sr_edm_block_grads* g, float* dzc,
                   float* de, char* scratch, hipStream_t st);

}  // namespace sr
