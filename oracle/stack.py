"""The sparse middle stack, the routed step and the dense mode.

Sparse middle stack (Eq. sparse_forward):  h_n2 = Block_n2 o ... o Block_1 (h0),
applied to the K routed tokens of every sample.  Dense mode (Sec. 3.4
"Architecture-agnostic design": r = 1 is the dense baseline): the same blocks
on all L tokens, no routing.

Routed step (Alg. 1, stage 2): select I, gather h0 = x[I], run the stack,
scatter x' = x0 + Scatter(h_n2 - h0, I).  Its backward follows from
x' = x0 + S(F(G x0) - G x0), with G the gather and S the scatter (S = G^T):
dx0 = g + S(J^T (G g) - G g), which is again a gather of g, the stack's VJP,
and a residual-delta scatter of (J^T g[I]) - g[I] into g.  Unselected rows
get dx0 = g exactly.

Precision reading: the stack runs in fp64 on the exact values of its storage
inputs.  Its output is rounded to the storage type once, at the end, before the
scatter (the HIP path keeps an fp32 residual stream inside the stack and rounds
at the same point).

Trunk (Sec. 3.2 "Three-stage block partition", Eq. partition): n1 dense early
blocks, the routed step on n2 middle blocks, n3 dense late blocks.  Each stage's
output is rounded to the storage type once (the dense stages' outputs and the
scatter's result are storage tensors on the HIP path too); the backward is the
late stage's VJP, the routed step's VJP and the early stage's VJP, with the same
roundings of the stage gradients.

Pins: keep = 100% with I = 0..L-1 equals the dense stack (fp64, to rounding);
unselected rows bit-identical; zero-initialised residual branches make x' == x
bit for bit; per-sample independence.
"""
from __future__ import annotations

import numpy as np

from . import block as blk
from . import routing
from .numerics import storage_to_f64, f64_to_storage


def params_f64(params):
    return [{k: storage_to_f64(v) for k, v in p.items()} for p in params]


def stack_fwd(h, params64, H, eps, kind="preln", cond=None, keep_cache=True, last_rows=None):
    """h: (B, S, D) fp64.  Returns (h_out fp64, caches).  ``last_rows`` evaluates only
    those query rows of the last block (sampled-output checks at full size)."""
    caches = []
    n = len(params64)
    for i, p in enumerate(params64):
        rows = last_rows if (i == n - 1) else None
        h, c = blk.block_fwd(h, p, H, eps, kind, cond, rows=rows)
        if keep_cache:
            caches.append(c)
    return h, caches


def stack_bwd(dh, params64, caches):
    """Returns (dh_in, grads per block, dcond summed over blocks or None)."""
    grads = [None] * len(params64)
    dcond = None
    for i in reversed(range(len(params64))):
        dh, g, dc = blk.block_bwd(dh, params64[i], caches[i])
        grads[i] = g
        if dc is not None:
            dcond = dc if dcond is None else dcond + dc
    return dh, grads, dcond


def routed_forward(x, idx, params, H, eps, kind="preln", cond=None, shared=False):
    """x: (B, L, D) storage.  Returns (x' storage, h0 storage, h_out fp64, h_out storage, caches)."""
    dtype = "bf16" if np.asarray(x).dtype == np.uint16 else "f32"
    h0 = routing.gather(x, idx, shared)
    p64 = params_f64(params)
    c64 = None if cond is None else storage_to_f64(cond)
    h_out, caches = stack_fwd(storage_to_f64(h0), p64, H, eps, kind, c64)
    h_out_s = f64_to_storage(h_out, dtype)
    x_new = routing.scatter_delta(x, h_out_s, h0, idx, shared)
    return x_new, h0, h_out, h_out_s, caches


def routed_backward(g, idx, params, caches, shared=False):
    """g: (B, L, D) storage upstream gradient.  Returns (dx0 storage, dh_in fp64, grads, dcond)."""
    dtype = "bf16" if np.asarray(g).dtype == np.uint16 else "f32"
    gh = routing.gather(g, idx, shared)
    p64 = params_f64(params)
    dh_in, grads, dcond = stack_bwd(storage_to_f64(gh), p64, caches)
    dx0 = routing.scatter_delta(g, f64_to_storage(dh_in, dtype), gh, idx, shared)
    return dx0, dh_in, grads, dcond


def dense_forward(x, params, H, eps, kind="preln", cond=None):
    p64 = params_f64(params)
    c64 = None if cond is None else storage_to_f64(cond)
    return stack_fwd(storage_to_f64(x), p64, H, eps, kind, c64)


def trunk_forward(x0, idx, params, split, H, eps):
    """x0: (B, L, D) storage; params: n1 + n2 + n3 blocks (early, middle, late).
    Returns (x3 fp64, caches of the three stages)."""
    n1, n2, n3 = split
    assert len(params) == n1 + n2 + n3
    dtype = "bf16" if np.asarray(x0).dtype == np.uint16 else "f32"
    x1, c_early = dense_forward(x0, params[:n1], H, eps)
    x2, _, _, _, c_mid = routed_forward(f64_to_storage(x1, dtype), idx, params[n1:n1 + n2], H, eps)
    x3, c_late = dense_forward(x2, params[n1 + n2:], H, eps)
    return x3, (c_early, c_mid, c_late)


def trunk_backward(g3, idx, params, split, caches):
    """g3: (B, L, D) storage gradient of the trunk output.  Returns (g0 fp64, grads of
    all n1 + n2 + n3 blocks in trunk order)."""
    n1, n2, n3 = split
    dtype = "bf16" if np.asarray(g3).dtype == np.uint16 else "f32"
    c_early, c_mid, c_late = caches
    g2, gr_late, _ = stack_bwd(storage_to_f64(g3), params_f64(params[n1 + n2:]), c_late)
    g1, _, gr_mid, _ = routed_backward(f64_to_storage(g2, dtype), idx, params[n1:n1 + n2], c_mid)
    g0, gr_early, _ = stack_bwd(storage_to_f64(g1), params_f64(params[:n1]), c_early)
    return g0, gr_early + gr_mid + gr_late
