"""The generative model's block with the asymmetric attention of the sparse middle stage
(Sec. 3.4 "Integration with Generative Forecasting", Alg. 2; Sec. 3.1 "Generative
forecasting"; App. A.1, EDM architecture table), forward and backward in fp64.

Test infrastructure: this is the oracle; nothing on the product path imports it.

The paper gives the block's parts in order -- FiLM modulation (scale, shift from the noise
embedding e), self-attention, cross-attention to the conditioning sequence Z_c gated by
sigmoid(W e), MLP -- but not their equations.  The reading taken here:

    (shift, scale) = e W_film^T + b_film                       per sample, 2D values
    u   = LN0(h) * (1 + scale) + shift                          LN0: LayerNorm without affine
    h1  = h + SelfAttn(u)                                       the S tokens of h only
    g   = sigmoid(e W_g^T + b_g)                                per sample and channel
    h2  = h1 + g * CrossAttn(LNc(h1), Z_c)
    h'  = h2 + MLP(LN2(h2))

SelfAttn and MLP are those of the pre-LN block (oracle/block.py).  CrossAttn(x, Z):
q = x W_q^T + b_q (the S query tokens), [k v] = Z W_kv^T + b_kv (all L conditioning
tokens, rows of W_kv ordered k, v, head-major within each), per head
P = softmax(q k^T / sqrt(hd)) over the L keys, output (P v) W_oc^T + b_oc.  In the sparse
middle stage S = K routed tokens while Z_c keeps its L tokens: the asymmetry of Sec. 3.4,
cost O(K L D) instead of O(L^2 D).

Backward: the vector-Jacobian products written out by hand, as in oracle/block.py, plus
sigmoid'(x) = s (1 - s).  It returns the gradients of h, of every parameter, of Z_c and of
e (Z_c and e are shared by all blocks, so a stack sums theirs).

Pins (tests/test_oracle_edm_block.py): torch CPU fp64 autograd of the same block from
torch.nn.functional primitives; central finite differences; a closed gate (sigmoid -> 0)
makes the output independent of Z_c with dZ_c = 0; one conditioning token makes every
query's cross-attention output that token's value; cross-attention rows are independent of
the other queries (the routed block's cross-attention rows are the dense block's rows).
"""
from __future__ import annotations

import numpy as np
from scipy.special import expit

from .block import (attention_bwd, attention_fwd, gelu, gelu_grad, ln_bwd, ln_fwd, merge_heads,
                    split_heads)

EDM_PARAM_NAMES = (
    "w_film", "b_film", "w_qkv", "b_qkv", "w_o", "b_o",
    "lnc_w", "lnc_b", "w_q", "b_q", "w_kv", "b_kv", "w_oc", "b_oc", "w_g", "b_g",
    "ln2_w", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2",
)


def edm_block_fwd(h, zc, e, p, H, eps):
    """h: (B, S, D) tokens; zc: (B, L, D) conditioning tokens; e: (B, D) noise embedding;
    p: dict of fp64 parameters ([out, in] weights).  Returns (h_out, cache)."""
    B, S, D = h.shape
    film = e @ p["w_film"].T + p["b_film"]                       # (B, 2D)
    shift, scale = film[:, None, :D], film[:, None, D:]
    n0, c_ln0 = ln_fwd(h, None, None, eps)
    u = n0 * (1.0 + scale) + shift
    qkv = u @ p["w_qkv"].T + p["b_qkv"]
    q = split_heads(qkv[..., :D], H)
    k = split_heads(qkv[..., D:2 * D], H)
    v = split_heads(qkv[..., 2 * D:], H)
    O = merge_heads(attention_fwd(q, k, v))
    h1 = h + O @ p["w_o"].T + p["b_o"]

    uc, c_lnc = ln_fwd(h1, p["lnc_w"], p["lnc_b"], eps)
    qc = split_heads(uc @ p["w_q"].T + p["b_q"], H)              # (B, H, S, hd)
    kv = zc @ p["w_kv"].T + p["b_kv"]                            # (B, L, 2D)
    kc = split_heads(kv[..., :D], H)                             # (B, H, L, hd)
    vc = split_heads(kv[..., D:], H)
    Oc = merge_heads(attention_fwd(qc, kc, vc))                  # (B, S, D)
    c_out = Oc @ p["w_oc"].T + p["b_oc"]
    g = expit(e @ p["w_g"].T + p["b_g"])                         # sigmoid, (B, D)
    h2 = h1 + g[:, None, :] * c_out

    u2, c_ln2 = ln_fwd(h2, p["ln2_w"], p["ln2_b"], eps)
    z = u2 @ p["w_fc1"].T + p["b_fc1"]
    gz = gelu(z)
    h_out = h2 + gz @ p["w_fc2"].T + p["b_fc2"]
    cache = dict(H=H, e=e, zc=zc, n0=n0, c_ln0=c_ln0, scale=scale, u=u, q=q, k=k, v=v, O=O,
                 uc=uc, c_lnc=c_lnc, qc=qc, kc=kc, vc=vc, Oc=Oc, c_out=c_out, g=g,
                 u2=u2, c_ln2=c_ln2, z=z, gz=gz)
    return h_out, cache


def edm_block_bwd(dh_out, p, cache):
    """Returns (dh_in, grads dict over EDM_PARAM_NAMES, dzc, de)."""
    H = cache["H"]
    grads = {}
    dsum = lambda t: t.sum(axis=(0, 1))
    flat = lambda t: t.reshape(-1, t.shape[-1])

    # MLP
    grads["w_fc2"] = flat(dh_out).T @ flat(cache["gz"])
    grads["b_fc2"] = dsum(dh_out)
    dz = (dh_out @ p["w_fc2"]) * gelu_grad(cache["z"])
    grads["w_fc1"] = flat(dz).T @ flat(cache["u2"])
    grads["b_fc1"] = dsum(dz)
    dx, grads["ln2_w"], grads["ln2_b"] = ln_bwd(dz @ p["w_fc1"], cache["c_ln2"], p["ln2_w"])
    dh2 = dh_out + dx

    # gated cross-attention
    g = cache["g"]
    dc = dh2 * g[:, None, :]
    dglog = (dh2 * cache["c_out"]).sum(axis=1) * g * (1.0 - g)   # (B, D)
    grads["w_g"] = dglog.T @ cache["e"]
    grads["b_g"] = dglog.sum(axis=0)
    de = dglog @ p["w_g"]
    grads["w_oc"] = flat(dc).T @ flat(cache["Oc"])
    grads["b_oc"] = dsum(dc)
    dqc, dkc, dvc = attention_bwd(cache["qc"], cache["kc"], cache["vc"], split_heads(dc @ p["w_oc"], H))
    dq_lin = merge_heads(dqc)
    grads["w_q"] = flat(dq_lin).T @ flat(cache["uc"])
    grads["b_q"] = dsum(dq_lin)
    dkv = np.concatenate([merge_heads(dkc), merge_heads(dvc)], axis=-1)   # (B, L, 2D)
    grads["w_kv"] = flat(dkv).T @ flat(cache["zc"])
    grads["b_kv"] = dsum(dkv)
    dzc = dkv @ p["w_kv"]
    dx, grads["lnc_w"], grads["lnc_b"] = ln_bwd(dq_lin @ p["w_q"], cache["c_lnc"], p["lnc_w"])
    dh1 = dh2 + dx

    # FiLM-modulated self-attention
    grads["w_o"] = flat(dh1).T @ flat(cache["O"])
    grads["b_o"] = dsum(dh1)
    dq, dk, dv = attention_bwd(cache["q"], cache["k"], cache["v"], split_heads(dh1 @ p["w_o"], H))
    dqkv = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)], axis=-1)
    grads["w_qkv"] = flat(dqkv).T @ flat(cache["u"])
    grads["b_qkv"] = dsum(dqkv)
    du = dqkv @ p["w_qkv"]
    dfilm = np.concatenate([du.sum(axis=1), (du * cache["n0"]).sum(axis=1)], axis=-1)   # (B, 2D): shift, scale
    grads["w_film"] = dfilm.T @ cache["e"]
    grads["b_film"] = dfilm.sum(axis=0)
    de = de + dfilm @ p["w_film"]
    dx, _, _ = ln_bwd(du * (1.0 + cache["scale"]), cache["c_ln0"], None)
    return dh1 + dx, grads, dzc, de
