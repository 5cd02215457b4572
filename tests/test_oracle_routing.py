"""Pins of the oracle's gather / residual-delta scatter (Eq. scatter) and of the
routed stack (Alg. 1 stage 2; Sec. 3.4 dense mode)."""
import numpy as np
import pytest

from oracle import routing, stack, select
from oracle.numerics import f32_to_bf16_bits, bf16_bits_to_f32, storage_to_f64
from paper_2607_02829_amd import inputs

pytestmark = pytest.mark.cpu


def _bf16(a):
    return f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def test_gather_is_indexing():
    rng = np.random.default_rng(0)
    x = _bf16(rng.standard_normal((2, 20, 8)))
    idx = np.array([[1, 4, 19], [0, 2, 3]], dtype=np.int32)
    g = routing.gather(x, idx)
    assert np.array_equal(g[0], x[0, [1, 4, 19]]) and np.array_equal(g[1], x[1, [0, 2, 3]])
    gs = routing.gather(x, idx[:1], shared=True)
    assert np.array_equal(gs[1], x[1, [1, 4, 19]])


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_unselected_rows_bit_identical(dt):
    rng = np.random.default_rng(1)
    B, L, K, D = 2, 40, 10, 16
    x = inputs.to_storage(rng.standard_normal((B, L, D)), dt)
    idx = select.select_random(B, L, K, 1, 0)
    h0 = routing.gather(x, idx)
    h = inputs.to_storage(rng.standard_normal((B, K, D)), dt)
    out = routing.scatter_delta(x, h, h0, idx)
    for b in range(B):
        mask = np.ones(L, bool); mask[idx[b]] = False
        assert np.array_equal(out[b, mask].view(np.uint8), x[b, mask].view(np.uint8))
    # h == h0 leaves everything bit-identical
    same = routing.scatter_delta(x, h0, h0, idx)
    assert np.array_equal(same.view(np.uint8), x.view(np.uint8))
    # omitting h0 re-reads x[idx], which is h0 by definition
    assert np.array_equal(routing.scatter_delta(x, h, None, idx), out)


def test_scatter_single_rounding_hand_case():
    # x0 = 1, h0 = 1 + 2^-7 (bf16 neighbour), h = 1 + 2^-6: delta = 2^-7 exactly in fp32,
    # x' = 1 + 2^-7 exactly representable.  With x0 = 256, delta 2^-7 is below half an
    # ulp of bf16 at 256 (ulp = 2), so x' rounds back to 256.
    x = _bf16([[[1.0], [256.0]]])
    idx = np.array([[0, 1]], dtype=np.int32)
    h0 = _bf16([[[1.0 + 2 ** -7], [1.0 + 2 ** -7]]])
    h = _bf16([[[1.0 + 2 ** -6], [1.0 + 2 ** -6]]])
    out = bf16_bits_to_f32(routing.scatter_delta(x, h, h0, idx))
    assert out[0, 0, 0] == np.float32(1.0 + 2 ** -7)
    assert out[0, 1, 0] == np.float32(256.0)
    # 1 + (1 + 2^-7) = 2 + 2^-7 exactly in fp32; at 2 the bf16 ulp is 2^-6, so this is a tie -> even (2.0)
    x2 = _bf16([[[1.0]]]); h0b = _bf16([[[0.0]]]); hb = _bf16([[[1.0 + 2 ** -7]]])
    out2 = bf16_bits_to_f32(routing.scatter_delta(x2, hb, h0b, np.array([[0]], np.int32)))
    assert out2[0, 0, 0] == np.float32(2.0)


def _wl(**kw):
    return inputs.small(**kw)


@pytest.mark.parametrize("kind", ["preln", "adaln"])
def test_zero_branches_scatter_is_identity(kind):
    w = _wl(D=32, H=2, F=128, n_blocks=2, kind=kind)
    x = inputs.to_storage(inputs.token_field(w), "bf16")
    zero = ("w_ada", "b_ada") if kind == "adaln" else ("w_o", "b_o", "w_fc2", "b_fc2")
    params = inputs.params_to_storage(inputs.block_params(w, zero=zero), "bf16")
    cond = inputs.to_storage(inputs.cond_vector(w), "bf16") if kind == "adaln" else None
    idx = select.select_random(w.B, w.L, w.K, 42, 0)
    x_new, *_ = stack.routed_forward(x, idx, params, w.H, 1e-6, kind, cond)
    assert np.array_equal(x_new, x)


def test_keep_all_equals_dense():
    w = _wl(D=32, H=2, F=128, n_blocks=2)
    x = inputs.to_storage(inputs.token_field(w), "bf16")
    params = inputs.params_to_storage(inputs.block_params(w, randomise_affine=True), "bf16")
    idx = np.tile(np.arange(w.L, dtype=np.int32), (w.B, 1))
    _, _, h_routed, _, _ = stack.routed_forward(x, idx, params, w.H, 1e-6)
    h_dense, _ = stack.dense_forward(x, params, w.H, 1e-6)
    np.testing.assert_allclose(h_routed, h_dense, rtol=1e-12, atol=1e-12)


def test_per_sample_independence():
    w = _wl(D=32, H=2, F=128, n_blocks=2)
    x = inputs.to_storage(inputs.token_field(w), "bf16")
    params = inputs.params_to_storage(inputs.block_params(w), "bf16")
    idx = select.select_random(w.B, w.L, w.K, 42, 0)
    a, *_ = stack.routed_forward(x, idx, params, w.H, 1e-6)
    x2 = x.copy(); x2[1] = x2[1][::-1]
    b, *_ = stack.routed_forward(x2, idx, params, w.H, 1e-6)
    assert np.array_equal(a[0], b[0])


def test_routed_backward_unselected_rows_pass_through():
    w = _wl(D=32, H=2, F=128, n_blocks=1)
    x = inputs.to_storage(inputs.token_field(w), "bf16")
    params = inputs.params_to_storage(inputs.block_params(w), "bf16")
    idx = select.select_random(w.B, w.L, w.K, 42, 0)
    _, _, _, _, caches = stack.routed_forward(x, idx, params, w.H, 1e-6)
    g = inputs.to_storage(inputs.upstream_grad(w), "bf16")
    dx0, dh_in, grads, _ = stack.routed_backward(g, idx, params, caches)
    for b in range(w.B):
        mask = np.ones(w.L, bool); mask[idx[b]] = False
        assert np.array_equal(dx0[b, mask], g[b, mask])


def test_routed_backward_is_vjp_of_routed_forward():
    # fp32 storage; compare the routed VJP to central differences of the fp64 map
    # x0 -> x0 + S(F(G x0) - G x0) (storage rounding left out of the differenced map).
    w = _wl(D=8, H=2, F=32, n_blocks=1, B=1, Hg=3, Wg=4, keep=0.5)
    rng = np.random.default_rng(3)
    x = rng.standard_normal((w.B, w.L, w.D))
    p = stack.params_f64(inputs.block_params(w, randomise_affine=True, std=0.3))
    idx = select.select_random(w.B, w.L, w.K, 1, 0)
    g = rng.standard_normal((w.B, w.L, w.D))

    def fwd(x_):
        h0 = x_[:, idx[0], :]
        h, c = stack.stack_fwd(h0, p, w.H, 1e-6)
        out = x_.copy(); out[:, idx[0], :] += h - h0
        return out, c

    _, caches = fwd(x)
    dh_in, _, _ = stack.stack_bwd(g[:, idx[0], :], p, caches)
    dx = g.copy(); dx[:, idx[0], :] += dh_in - g[:, idx[0], :]
    for fi in range(0, x.size, 7):
        ix = np.unravel_index(fi, x.shape)
        e = 1e-6
        a = x.copy(); a[ix] += e
        b = x.copy(); b[ix] -= e
        num = ((fwd(a)[0] - fwd(b)[0]) * g).sum() / (2 * e)
        assert abs(num - dx[ix]) < 1e-6 * max(1, abs(num))
