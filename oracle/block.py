"""One middle block, forward and backward, in fp64 (Sec. 3.3 block equation;
architecture tables in App. A.1).

Pre-LN ViT block (the deterministic model's block, Sec. 3.3):

    h1 = h  + SelfAttn(LN1(h))
    h' = h1 + MLP(LN2(h1))

LN(v) = (v - mean(v)) / sqrt(var(v) + eps) * gamma + beta, biased variance
over the D channels.  SelfAttn: [q k v] = u W_qkv^T + b_qkv (rows of W_qkv
ordered q, k, v; head j owns rows j*hd .. j*hd+hd-1 of each), per sample and
head P = softmax(q k^T / sqrt(hd)) over all S tokens (no mask, no positional
term inside the block), O = P v, heads concatenated, then O W_o^T + b_o.
MLP: GELU(u W_1^T + b_1) W_2^T + b_2, exact GELU(z) = z * Phi(z), hidden width
F = 4D (MLP ratio 4, App. A.1), dropout 0.

adaLN-modulated block (the diffusion workload's block; the paper's EDM block
conditions with FiLM scale/shift and a gate computed from a global vector,
Sec. 2 "Generative forecasting" and App. A.1 EDM table):

    (shift1, scale1, gate1, shift2, scale2, gate2) = c W_ada^T + b_ada   (per sample)
    h1 = h  + gate1 * SelfAttn(LN0(h)  * (1 + scale1) + shift1)
    h' = h1 + gate2 * MLP    (LN0(h1) * (1 + scale2) + shift2)

LN0 is LayerNorm without affine parameters.

Backward: the vector-Jacobian products of the above, written out by hand
(linear: dX = dY W, dW = dY^T X, db = sum dY; LN; GELU'(z) = Phi(z) + z phi(z);
softmax attention: dV = P^T dO, dP = dO V^T, dS = P o (dP - rowsum(P o dP)),
dQ = dS K / sqrt(hd), dK = dS^T Q / sqrt(hd)).

Pins (tests/test_oracle_block.py): cross-check against torch CPU fp64 autograd
of the same block built from torch.nn.functional primitives; central finite
differences on tiny shapes for every input and parameter; S = 1 gives O = v;
W_q = b_q = 0 gives uniform attention; zero W_o, b_o, W_2, b_2 (adaLN: zero
W_ada, b_ada) gives the identity; permutation equivariance over tokens.
"""
from __future__ import annotations

import math

import numpy as np
from scipy.special import erf

SQRT2 = math.sqrt(2.0)
INV_SQRT_2PI = 1.0 / math.sqrt(2.0 * math.pi)


# ----------------------------------------------------------------------------- pieces

def ln_fwd(x, gamma, beta, eps):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mu) * rstd
    y = xhat if gamma is None else xhat * gamma + beta
    return y, (xhat, rstd)


def ln_bwd(dy, cache, gamma):
    xhat, rstd = cache
    dxhat = dy if gamma is None else dy * gamma
    m1 = dxhat.mean(axis=-1, keepdims=True)
    m2 = (dxhat * xhat).mean(axis=-1, keepdims=True)
    dx = (dxhat - m1 - xhat * m2) * rstd
    dgamma = (dy * xhat).sum(axis=(0, 1))
    dbeta = dy.sum(axis=(0, 1))
    return dx, dgamma, dbeta


def gelu(z):
    return 0.5 * z * (1.0 + erf(z / SQRT2))


def gelu_grad(z):
    return 0.5 * (1.0 + erf(z / SQRT2)) + z * INV_SQRT_2PI * np.exp(-0.5 * z * z)


def softmax_rows(s):
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    return e / e.sum(axis=-1, keepdims=True)


def split_heads(t, H):
    B, S, D = t.shape
    return t.reshape(B, S, H, D // H).transpose(0, 2, 1, 3)       # (B, H, S, hd)


def merge_heads(t):
    B, H, S, hd = t.shape
    return t.transpose(0, 2, 1, 3).reshape(B, S, H * hd)


def attention_fwd(q, k, v, rows=None):
    """q, k, v: (B, H, S, hd).  Returns O (B, H, S', hd) for query rows ``rows`` (all if None)."""
    B, H, S, hd = q.shape
    scale = 1.0 / math.sqrt(hd)
    qr = q if rows is None else q[:, :, rows, :]
    out = np.empty(qr.shape, dtype=np.float64)
    for b in range(B):
        for j in range(H):
            P = softmax_rows(qr[b, j] @ k[b, j].T * scale)
            out[b, j] = P @ v[b, j]
    return out


def attention_bwd(q, k, v, dO):
    B, H, S, hd = q.shape
    scale = 1.0 / math.sqrt(hd)
    dq = np.empty_like(q)
    dk = np.empty_like(k)
    dv = np.empty_like(v)
    for b in range(B):
        for j in range(H):
            P = softmax_rows(q[b, j] @ k[b, j].T * scale)
            dv[b, j] = P.T @ dO[b, j]
            dP = dO[b, j] @ v[b, j].T
            dS = P * (dP - (P * dP).sum(axis=-1, keepdims=True))
            dq[b, j] = dS @ k[b, j] * scale
            dk[b, j] = dS.T @ q[b, j] * scale
    return dq, dk, dv


# ----------------------------------------------------------------------------- block

def _mod_chunks(p, cond):
    mod = cond @ p["w_ada"].T + p["b_ada"]                        # (B, 6D)
    D = cond.shape[1]
    return [mod[:, i * D:(i + 1) * D][:, None, :] for i in range(6)], mod


def block_fwd(h, p, H, eps, kind="preln", cond=None, rows=None):
    """h: (B, S, D) fp64; p: dict of fp64 parameters.

    Returns (h_out, cache).  With ``rows`` (query-row indices), h_out holds only
    those rows and no cache is returned (attention keys and values still span
    all S tokens)."""
    B, S, D = h.shape
    if kind == "adaln":
        (sh1, sc1, g1, sh2, sc2, g2), _ = _mod_chunks(p, cond)
        n1, c_ln1 = ln_fwd(h, None, None, eps)
        u = n1 * (1.0 + sc1) + sh1
    else:
        u, c_ln1 = ln_fwd(h, p["ln1_w"], p["ln1_b"], eps)
    qkv = u @ p["w_qkv"].T + p["b_qkv"]
    q = split_heads(qkv[..., :D], H)
    k = split_heads(qkv[..., D:2 * D], H)
    v = split_heads(qkv[..., 2 * D:], H)
    O = merge_heads(attention_fwd(q, k, v, rows))
    a_out = O @ p["w_o"].T + p["b_o"]
    hr = h if rows is None else h[:, rows, :]
    h1 = hr + (g1 * a_out if kind == "adaln" else a_out)
    if kind == "adaln":
        n2, c_ln2 = ln_fwd(h1, None, None, eps)
        u2 = n2 * (1.0 + sc2) + sh2
    else:
        u2, c_ln2 = ln_fwd(h1, p["ln2_w"], p["ln2_b"], eps)
    z = u2 @ p["w_fc1"].T + p["b_fc1"]
    gz = gelu(z)
    m_out = gz @ p["w_fc2"].T + p["b_fc2"]
    h_out = h1 + (g2 * m_out if kind == "adaln" else m_out)
    if rows is not None:
        return h_out, None
    cache = dict(h=h, u=u, c_ln1=c_ln1, q=q, k=k, v=v, O=O, a_out=a_out, h1=h1, u2=u2,
                 c_ln2=c_ln2, z=z, gz=gz, m_out=m_out, cond=cond, kind=kind, H=H)
    if kind == "adaln":
        cache.update(n1=c_ln1[0], n2=c_ln2[0], sc1=sc1, sc2=sc2, g1=g1, g2=g2)
    return h_out, cache


def block_bwd(dh_out, p, cache):
    """Returns (dh_in, grads dict with every parameter name, dcond or None)."""
    kind = cache["kind"]
    H = cache["H"]
    grads = {k: np.zeros_like(v) for k, v in p.items()}
    dsum = lambda t: t.sum(axis=(0, 1))
    flat = lambda t: t.reshape(-1, t.shape[-1])

    # MLP branch
    if kind == "adaln":
        dm = dh_out * cache["g2"]
        dgate2 = (dh_out * cache["m_out"]).sum(axis=1)
    else:
        dm = dh_out
    grads["w_fc2"] = flat(dm).T @ flat(cache["gz"])
    grads["b_fc2"] = dsum(dm)
    dgz = dm @ p["w_fc2"]
    dz = dgz * gelu_grad(cache["z"])
    grads["w_fc1"] = flat(dz).T @ flat(cache["u2"])
    grads["b_fc1"] = dsum(dz)
    du2 = dz @ p["w_fc1"]
    if kind == "adaln":
        dscale2 = (du2 * cache["n2"]).sum(axis=1)
        dshift2 = du2.sum(axis=1)
        dx, _, _ = ln_bwd(du2 * (1.0 + cache["sc2"]), cache["c_ln2"], None)
    else:
        dx, grads["ln2_w"], grads["ln2_b"] = ln_bwd(du2, cache["c_ln2"], p["ln2_w"])
    dh1 = dh_out + dx

    # attention branch
    if kind == "adaln":
        da = dh1 * cache["g1"]
        dgate1 = (dh1 * cache["a_out"]).sum(axis=1)
    else:
        da = dh1
    grads["w_o"] = flat(da).T @ flat(cache["O"])
    grads["b_o"] = dsum(da)
    dO = split_heads(da @ p["w_o"], H)
    dq, dk, dv = attention_bwd(cache["q"], cache["k"], cache["v"], dO)
    dqkv = np.concatenate([merge_heads(dq), merge_heads(dk), merge_heads(dv)], axis=-1)
    grads["w_qkv"] = flat(dqkv).T @ flat(cache["u"])
    grads["b_qkv"] = dsum(dqkv)
    du = dqkv @ p["w_qkv"]
    dcond = None
    if kind == "adaln":
        dscale1 = (du * cache["n1"]).sum(axis=1)
        dshift1 = du.sum(axis=1)
        dx, _, _ = ln_bwd(du * (1.0 + cache["sc1"]), cache["c_ln1"], None)
        dmod = np.concatenate([dshift1, dscale1, dgate1, dshift2, dscale2, dgate2], axis=-1)  # (B, 6D)
        grads["w_ada"] = dmod.T @ cache["cond"]
        grads["b_ada"] = dmod.sum(axis=0)
        dcond = dmod @ p["w_ada"]
    else:
        dx, grads["ln1_w"], grads["ln1_b"] = ln_bwd(du, cache["c_ln1"], p["ln1_w"])
    dh_in = dh1 + dx
    return dh_in, grads, dcond
