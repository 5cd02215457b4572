"""Pins of the oracle's generative block with asymmetric attention (Sec. 3.4 "Integration
with Generative Forecasting"; App. A.1 EDM table): S query tokens, L conditioning tokens."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import edm_block as eb

pytestmark = pytest.mark.cpu

EPS = 1e-6


def _params(D, F, rng):
    r = lambda *s: 0.3 * rng.standard_normal(s)
    return {
        "w_film": r(2 * D, D), "b_film": 0.1 * rng.standard_normal(2 * D),
        "w_qkv": r(3 * D, D), "b_qkv": 0.1 * rng.standard_normal(3 * D),
        "w_o": r(D, D), "b_o": 0.1 * rng.standard_normal(D),
        "lnc_w": 1 + 0.1 * rng.standard_normal(D), "lnc_b": 0.1 * rng.standard_normal(D),
        "w_q": r(D, D), "b_q": 0.1 * rng.standard_normal(D),
        "w_kv": r(2 * D, D), "b_kv": 0.1 * rng.standard_normal(2 * D),
        "w_oc": r(D, D), "b_oc": 0.1 * rng.standard_normal(D),
        "w_g": r(D, D), "b_g": 0.1 * rng.standard_normal(D),
        "ln2_w": 1 + 0.1 * rng.standard_normal(D), "ln2_b": 0.1 * rng.standard_normal(D),
        "w_fc1": r(F, D), "b_fc1": 0.1 * rng.standard_normal(F),
        "w_fc2": r(D, F), "b_fc2": 0.1 * rng.standard_normal(D),
    }


def _torch_block(h, zc, e, p, H):
    """The same block from torch.nn.functional primitives (independent implementation)."""
    B, S, D = h.shape
    L = zc.shape[1]
    heads = lambda t, n: t.reshape(B, n, H, D // H).transpose(1, 2)
    merge = lambda t, n: t.transpose(1, 2).reshape(B, n, D)
    shift, scale = Fn.linear(e, p["w_film"], p["b_film"])[:, None, :].chunk(2, dim=-1)
    u = Fn.layer_norm(h, (D,), eps=EPS) * (1 + scale) + shift
    q, k, v = Fn.linear(u, p["w_qkv"], p["b_qkv"]).chunk(3, dim=-1)
    o = merge(Fn.scaled_dot_product_attention(heads(q, S), heads(k, S), heads(v, S)), S)
    h1 = h + Fn.linear(o, p["w_o"], p["b_o"])
    qc = Fn.linear(Fn.layer_norm(h1, (D,), p["lnc_w"], p["lnc_b"], eps=EPS), p["w_q"], p["b_q"])
    kc, vc = Fn.linear(zc, p["w_kv"], p["b_kv"]).chunk(2, dim=-1)
    oc = merge(Fn.scaled_dot_product_attention(heads(qc, S), heads(kc, L), heads(vc, L)), S)
    gate = torch.sigmoid(Fn.linear(e, p["w_g"], p["b_g"]))[:, None, :]
    h2 = h1 + gate * Fn.linear(oc, p["w_oc"], p["b_oc"])
    u2 = Fn.layer_norm(h2, (D,), p["ln2_w"], p["ln2_b"], eps=EPS)
    return h2 + Fn.linear(Fn.gelu(Fn.linear(u2, p["w_fc1"], p["b_fc1"])), p["w_fc2"], p["b_fc2"])


def _inputs(B=2, S=5, L=13, D=16, F=64, seed=0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((B, S, D)), rng.standard_normal((B, L, D)), rng.standard_normal((B, D)),
            _params(D, F, rng), rng.standard_normal((B, S, D)))


@pytest.mark.parametrize("S,L", [(5, 13), (13, 5), (1, 7), (6, 1)])
def test_edm_block_matches_torch_autograd_fp64(S, L):
    H = 2
    h, zc, e, p, dy = _inputs(S=S, L=L)
    out, cache = eb.edm_block_fwd(h, zc, e, p, H, EPS)
    dh, grads, dzc, de = eb.edm_block_bwd(dy, p, cache)
    tp = {k: torch.tensor(v, requires_grad=True) for k, v in p.items()}
    th, tz, te = (torch.tensor(a, requires_grad=True) for a in (h, zc, e))
    tout = _torch_block(th, tz, te, tp, H)
    tout.backward(torch.tensor(dy))
    np.testing.assert_allclose(out, tout.detach().numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dh, th.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(dzc, tz.grad.numpy(), rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(de, te.grad.numpy(), rtol=1e-10, atol=1e-10)
    assert set(grads) == set(eb.EDM_PARAM_NAMES)
    for name, t in tp.items():
        np.testing.assert_allclose(grads[name], t.grad.numpy(), rtol=1e-10, atol=1e-10, err_msg=name)


def test_edm_block_finite_differences():
    H = 2
    h, zc, e, p, dy = _inputs(B=1, S=3, L=4, D=8, F=16, seed=3)
    f = lambda h_, z_, e_, p_: float((eb.edm_block_fwd(h_, z_, e_, p_, H, EPS)[0] * dy).sum())
    _, cache = eb.edm_block_fwd(h, zc, e, p, H, EPS)
    dh, grads, dzc, de = eb.edm_block_bwd(dy, p, cache)
    rng = np.random.default_rng(9)
    step = 1e-6

    def check(arr, grad, call):
        for _ in range(4):
            i = tuple(rng.integers(0, n) for n in arr.shape)
            old = arr[i]
            arr[i] = old + step; fp = call()
            arr[i] = old - step; fm = call()
            arr[i] = old
            assert abs((fp - fm) / (2 * step) - grad[i]) < 1e-6 * max(1.0, abs(grad[i]))

    call = lambda: f(h, zc, e, p)
    check(h, dh, call)
    check(zc, dzc, call)
    check(e, de, call)
    for name in ("w_film", "w_kv", "w_q", "w_g", "b_g", "lnc_w", "w_oc"):
        check(p[name], grads[name], call)


def test_closed_gate_cuts_the_conditioning():
    # sigmoid(-1e3) = 0 in fp64: the cross-attention contributes nothing and Z_c gets no gradient
    H = 2
    h, zc, e, p, dy = _inputs(seed=5)
    p["w_g"] = np.zeros_like(p["w_g"])
    p["b_g"] = np.full_like(p["b_g"], -1e3)
    a, cache = eb.edm_block_fwd(h, zc, e, p, H, EPS)
    b, _ = eb.edm_block_fwd(h, 3.0 * zc + 1.0, e, p, H, EPS)
    assert np.array_equal(a, b)
    _, grads, dzc, _ = eb.edm_block_bwd(dy, p, cache)
    assert not np.any(dzc) and not np.any(grads["w_kv"]) and not np.any(grads["w_q"])


def test_one_conditioning_token_gives_its_value():
    # softmax over a single key is 1: every query's cross-attention output is that token's
    # value projection, so h2 - h1 = g * ((z W_v^T + b_v) W_oc^T + b_oc) on every row
    H = 2
    h, zc, e, p, _ = _inputs(L=1, seed=6)
    D = h.shape[-1]
    _, c = eb.edm_block_fwd(h, zc, e, p, H, EPS)
    v = zc @ p["w_kv"][D:].T + p["b_kv"][D:]                       # (B, 1, D)
    want = v @ p["w_oc"].T + p["b_oc"]
    np.testing.assert_allclose(c["c_out"], np.broadcast_to(want, c["c_out"].shape), rtol=1e-12, atol=1e-12)


def test_cross_attention_rows_do_not_depend_on_other_queries():
    # the routed block's cross-attention keeps all L keys: for a query token, its
    # cross-attention output is the same whichever other tokens are routed with it
    H = 2
    h, zc, e, p, _ = _inputs(S=9, L=11, seed=8)
    _, full = eb.edm_block_fwd(h, zc, e, p, H, EPS)
    D = h.shape[-1]
    rows = np.array([1, 4, 8])
    # recompute the cross-attention of those rows from their h1 alone
    uc = (full["uc"][:, rows])
    q = uc @ p["w_q"].T + p["b_q"]
    kv = zc @ p["w_kv"].T + p["b_kv"]
    hd = D // H
    out = np.empty((h.shape[0], len(rows), D))
    for b in range(h.shape[0]):
        for j in range(H):
            s = q[b][:, j * hd:(j + 1) * hd] @ kv[b][:, j * hd:(j + 1) * hd].T / np.sqrt(hd)
            P = np.exp(s - s.max(axis=1, keepdims=True)); P /= P.sum(axis=1, keepdims=True)
            out[b][:, j * hd:(j + 1) * hd] = P @ kv[b][:, D + j * hd:D + (j + 1) * hd]
    np.testing.assert_allclose(out, full["Oc"][:, rows], rtol=1e-12, atol=1e-12)
