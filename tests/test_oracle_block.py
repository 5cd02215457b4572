"""Pins of the oracle's block forward/backward (Sec. 3.3 block equation)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import block as blk

pytestmark = pytest.mark.cpu

EPS = 1e-6


def _params(D, F, rng, kind="preln"):
    p = {
        "ln1_w": 1 + 0.1 * rng.standard_normal(D), "ln1_b": 0.1 * rng.standard_normal(D),
        "w_qkv": 0.3 * rng.standard_normal((3 * D, D)), "b_qkv": 0.1 * rng.standard_normal(3 * D),
        "w_o": 0.3 * rng.standard_normal((D, D)), "b_o": 0.1 * rng.standard_normal(D),
        "ln2_w": 1 + 0.1 * rng.standard_normal(D), "ln2_b": 0.1 * rng.standard_normal(D),
        "w_fc1": 0.3 * rng.standard_normal((F, D)), "b_fc1": 0.1 * rng.standard_normal(F),
        "w_fc2": 0.3 * rng.standard_normal((D, F)), "b_fc2": 0.1 * rng.standard_normal(D),
        "w_ada": 0.3 * rng.standard_normal((6 * D, D)), "b_ada": 0.1 * rng.standard_normal(6 * D),
    }
    return p


def _torch_block(h, p, H, kind, cond):
    """The same block from torch.nn.functional primitives (independent implementation)."""
    D = h.shape[-1]
    if kind == "adaln":
        mod = Fn.linear(cond, p["w_ada"], p["b_ada"])
        sh1, sc1, g1, sh2, sc2, g2 = [m[:, None, :] for m in mod.chunk(6, dim=-1)]
        u = Fn.layer_norm(h, (D,), eps=EPS) * (1 + sc1) + sh1
    else:
        u = Fn.layer_norm(h, (D,), p["ln1_w"], p["ln1_b"], eps=EPS)
    q, k, v = Fn.linear(u, p["w_qkv"], p["b_qkv"]).chunk(3, dim=-1)
    B, S, _ = h.shape
    sh = lambda t: t.reshape(B, S, H, D // H).transpose(1, 2)
    o = Fn.scaled_dot_product_attention(sh(q), sh(k), sh(v)).transpose(1, 2).reshape(B, S, D)
    a = Fn.linear(o, p["w_o"], p["b_o"])
    h1 = h + (g1 * a if kind == "adaln" else a)
    if kind == "adaln":
        u2 = Fn.layer_norm(h1, (D,), eps=EPS) * (1 + sc2) + sh2
    else:
        u2 = Fn.layer_norm(h1, (D,), p["ln2_w"], p["ln2_b"], eps=EPS)
    m = Fn.linear(Fn.gelu(Fn.linear(u2, p["w_fc1"], p["b_fc1"])), p["w_fc2"], p["b_fc2"])
    return h1 + (g2 * m if kind == "adaln" else m)


@pytest.mark.parametrize("kind", ["preln", "adaln"])
def test_block_matches_torch_autograd_fp64(kind):
    rng = np.random.default_rng(0)
    B, S, D, H, F = 2, 7, 16, 2, 64
    p = _params(D, F, rng)
    h = rng.standard_normal((B, S, D))
    cond = rng.standard_normal((B, D)) if kind == "adaln" else None
    dy = rng.standard_normal((B, S, D))

    out, cache = blk.block_fwd(h, p, H, EPS, kind, cond)
    dh, grads, dcond = blk.block_bwd(dy, p, cache)

    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items()}
    th = torch.tensor(h, requires_grad=True)
    tc = torch.tensor(cond, requires_grad=True) if cond is not None else None
    tout = _torch_block(th, tp, H, kind, tc)
    tout.backward(torch.tensor(dy))
    np.testing.assert_allclose(out, tout.detach().numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dh, th.grad.numpy(), rtol=1e-10, atol=1e-10)
    for name, t in tp.items():
        want = t.grad.numpy() if t.grad is not None else np.zeros_like(p[name])
        np.testing.assert_allclose(grads[name], want, rtol=1e-10, atol=1e-10, err_msg=name)
    if kind == "adaln":
        np.testing.assert_allclose(dcond, tc.grad.numpy(), rtol=1e-10, atol=1e-10)


@pytest.mark.parametrize("kind", ["preln", "adaln"])
def test_block_finite_differences(kind):
    rng = np.random.default_rng(1)
    B, S, D, H, F = 2, 5, 8, 2, 32
    p = _params(D, F, rng)
    h = rng.standard_normal((B, S, D))
    cond = rng.standard_normal((B, D)) if kind == "adaln" else None
    dy = rng.standard_normal((B, S, D))
    out, cache = blk.block_fwd(h, p, H, EPS, kind, cond)
    dh, grads, dcond = blk.block_bwd(dy, p, cache)

    def loss(h_, p_, c_):
        return float((blk.block_fwd(h_, p_, H, EPS, kind, c_)[0] * dy).sum())

    def fd(arr, setter, n=6):
        errs = []
        flat_idx = rng.choice(arr.size, size=min(n, arr.size), replace=False)
        for fi in flat_idx:
            ix = np.unravel_index(fi, arr.shape)
            e = 1e-6 * max(1.0, abs(arr[ix]))
            a1 = arr.copy(); a1[ix] += e
            a2 = arr.copy(); a2[ix] -= e
            errs.append((ix, (setter(a1) - setter(a2)) / (2 * e)))
        return errs

    def check(analytic, pairs, name):
        for ix, num in pairs:
            assert abs(analytic[ix] - num) <= 1e-6 * max(1.0, abs(num)), (name, ix, analytic[ix], num)

    check(dh, fd(h, lambda a: loss(a, p, cond)), "h")
    for name in p:
        if kind == "adaln" and name.startswith("ln"):
            assert not grads[name].any()
            continue
        if kind == "preln" and name in ("w_ada", "b_ada"):
            assert not grads[name].any()
            continue
        check(grads[name], fd(p[name], lambda a, n=name: loss(h, {**p, n: a}, cond)), name)
    if kind == "adaln":
        check(dcond, fd(cond, lambda a: loss(h, p, a)), "cond")


def test_attention_single_token_returns_v():
    rng = np.random.default_rng(2)
    q, k, v = (rng.standard_normal((2, 3, 1, 8)) for _ in range(3))
    assert np.array_equal(blk.attention_fwd(q, k, v), v)


def test_attention_zero_query_is_mean_of_values():
    rng = np.random.default_rng(3)
    k, v = (rng.standard_normal((1, 2, 9, 4)) for _ in range(2))
    q = np.zeros_like(k)
    out = blk.attention_fwd(q, k, v)
    np.testing.assert_allclose(out, np.broadcast_to(v.mean(axis=2, keepdims=True), v.shape), rtol=1e-14, atol=1e-14)


def test_attention_bruteforce_textbook():
    # softmax(q k^T / sqrt(hd)) v written with explicit loops
    rng = np.random.default_rng(4)
    q, k, v = (rng.standard_normal((1, 1, 5, 3)) for _ in range(3))
    out = blk.attention_fwd(q, k, v)[0, 0]
    for i in range(5):
        w = [math.exp(sum(q[0, 0, i, d] * k[0, 0, j, d] for d in range(3)) / math.sqrt(3)) for j in range(5)]
        want = [sum(w[j] * v[0, 0, j, d] for j in range(5)) / sum(w) for d in range(3)]
        np.testing.assert_allclose(out[i], want, rtol=1e-13)


@pytest.mark.parametrize("kind", ["preln", "adaln"])
def test_zero_residual_branches_give_identity(kind):
    rng = np.random.default_rng(5)
    D, F, H = 16, 64, 4
    p = _params(D, F, rng)
    if kind == "adaln":
        p["w_ada"][:] = 0; p["b_ada"][:] = 0               # gates are zero
    else:
        for n in ("w_o", "b_o", "w_fc2", "b_fc2"):
            p[n][:] = 0
    h = rng.standard_normal((2, 6, D))
    cond = rng.standard_normal((2, D)) if kind == "adaln" else None
    out, _ = blk.block_fwd(h, p, H, EPS, kind, cond)
    assert np.array_equal(out, h)


def test_permutation_equivariance():
    rng = np.random.default_rng(6)
    D, F, H = 16, 64, 4
    p = _params(D, F, rng)
    h = rng.standard_normal((1, 11, D))
    perm = rng.permutation(11)
    a, _ = blk.block_fwd(h, p, H, EPS)
    b, _ = blk.block_fwd(h[:, perm], p, H, EPS)
    np.testing.assert_allclose(a[:, perm], b, rtol=1e-12, atol=1e-12)


def test_sampled_rows_match_full():
    rng = np.random.default_rng(7)
    D, F, H = 16, 64, 4
    p = _params(D, F, rng)
    h = rng.standard_normal((2, 13, D))
    rows = np.array([0, 5, 12])
    full, _ = blk.block_fwd(h, p, H, EPS)
    part, _ = blk.block_fwd(h, p, H, EPS, rows=rows)
    np.testing.assert_allclose(part, full[:, rows], rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("Sq,Skv", [(5, 13), (13, 5), (1, 9), (7, 1)])
def test_attention_with_two_token_counts_matches_torch(Sq, Skv):
    # the oracle's attention with different query and key counts (the generative block's
    # asymmetric attention) against torch fp64 autograd of softmax(q k^T / sqrt(hd)) v
    rng = np.random.default_rng([Sq, Skv])
    B, H, hd = 2, 3, 8
    q = rng.standard_normal((B, H, Sq, hd))
    k = rng.standard_normal((B, H, Skv, hd))
    v = rng.standard_normal((B, H, Skv, hd))
    dO = rng.standard_normal((B, H, Sq, hd))
    out = blk.attention_fwd(q, k, v)
    dq, dk, dv = blk.attention_bwd(q, k, v, dO)
    tq, tk, tv = (torch.tensor(a, requires_grad=True) for a in (q, k, v))
    tout = torch.softmax(tq @ tk.transpose(-1, -2) / math.sqrt(hd), dim=-1) @ tv
    tout.backward(torch.tensor(dO))
    np.testing.assert_allclose(out, tout.detach().numpy(), rtol=1e-12, atol=1e-12)
    for a, t in ((dq, tq), (dk, tk), (dv, tv)):
        np.testing.assert_allclose(a, t.grad.numpy(), rtol=1e-10, atol=1e-10)
    # brute force on one (sample, head, query)
    s = [sum(q[1, 2, Sq - 1, d] * k[1, 2, j, d] for d in range(hd)) / math.sqrt(hd) for j in range(Skv)]
    e = [math.exp(x - max(s)) for x in s]
    want = [sum(e[j] * v[1, 2, j, d] for j in range(Skv)) / sum(e) for d in range(hd)]
    np.testing.assert_allclose(out[1, 2, Sq - 1], want, rtol=1e-12, atol=1e-12)
