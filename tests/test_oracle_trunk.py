"""Pins of the oracle's dense-sparse-dense trunk (Sec. 3.2 "Three-stage block
partition", Eq. partition, and the routed step of Alg. 1 between the two dense
stages), against dense stacks computed without any routing."""
import numpy as np
import pytest

from oracle import stack, select
from oracle.numerics import storage_to_f64
from paper_2607_02829_amd import inputs

pytestmark = pytest.mark.cpu

W = inputs.small("trunk", B=2, Hg=6, Wg=7, D=32, H=2, F=64, dtype="f32")


def _rel(a, b):
    return float(np.abs(a - b).max() / np.abs(b).max())


def _setup(split, zero_mid=False):
    n = sum(split)
    p32 = inputs.block_params(W, n, randomise_affine=True)
    if zero_mid:
        n1, n2, _ = split
        for p in p32[n1:n1 + n2]:
            for k in ("w_o", "b_o", "w_fc2", "b_fc2"):
                p[k] = np.zeros_like(p[k])
    params = inputs.params_to_storage(p32, "f32")
    x0 = inputs.to_storage(inputs.token_field(W), "f32")
    g3 = inputs.to_storage(inputs.upstream_grad(W), "f32")
    return params, x0, g3


@pytest.mark.parametrize("split", [(1, 1, 1), (2, 3, 1)])
def test_keep_all_equals_dense_stack_of_all_blocks(split):
    # I = 0..L-1: the trunk is the dense stack of its n1 + n2 + n3 blocks, forward and backward
    params, x0, g3 = _setup(split)
    idx = np.tile(np.arange(W.L, dtype=np.int32), (W.B, 1))
    x3, caches = stack.trunk_forward(x0, idx, params, split, W.H, 1e-6)
    ref, rc = stack.dense_forward(x0, params, W.H, 1e-6)
    assert _rel(x3, ref) < 1e-6
    g0, grads = stack.trunk_backward(g3, idx, params, split, caches)
    rg0, rgrads, _ = stack.stack_bwd(storage_to_f64(g3), stack.params_f64(params), rc)
    assert _rel(g0, rg0) < 1e-5
    for a, b in zip(grads, rgrads):
        for k in ("w_qkv", "w_o", "w_fc1", "w_fc2", "ln1_w", "b_fc2"):
            assert _rel(a[k], b[k]) < 1e-5, k


def test_zero_middle_branches_leave_early_and_late_stages():
    # middle blocks whose residual branches are zero add no delta: the trunk is the dense
    # stack of the early and late blocks alone, and the gradient reaches x0 through those only
    split = (2, 2, 1)
    params, x0, g3 = _setup(split, zero_mid=True)
    idx = select.select_random(W.B, W.L, 10, 3, 0)
    x3, caches = stack.trunk_forward(x0, idx, params, split, W.H, 1e-6)
    outer = params[:2] + params[4:]
    ref, rc = stack.dense_forward(x0, outer, W.H, 1e-6)
    assert _rel(x3, ref) < 1e-6
    g0, grads = stack.trunk_backward(g3, idx, params, split, caches)
    rg0, rgrads, _ = stack.stack_bwd(storage_to_f64(g3), stack.params_f64(outer), rc)
    assert _rel(g0, rg0) < 1e-5
    for a, b in zip(grads[:2] + grads[4:], rgrads):
        assert _rel(a["w_fc1"], b["w_fc1"]) < 1e-5


def test_unrouted_rows_see_only_dense_stages():
    # a row never routed keeps its early-stage value through the middle stage: changing the
    # middle blocks' weights changes x3 only through rows the late stage's attention mixes in,
    # so with a single dense late block of zero attention output the unrouted rows of x3 are
    # independent of the middle weights
    split = (1, 1, 1)
    params, x0, _ = _setup(split)
    for k in ("w_o", "b_o"):
        params[2][k] = np.zeros_like(params[2][k])
    idx = select.select_random(W.B, W.L, 9, 5, 1)
    a, _ = stack.trunk_forward(x0, idx, params, split, W.H, 1e-6)
    p2 = [dict(p) for p in params]
    p2[1]["w_fc2"] = (p2[1]["w_fc2"] * 3.0).astype(np.float32)
    b, _ = stack.trunk_forward(x0, idx, p2, split, W.H, 1e-6)
    for bb in range(W.B):
        mask = np.ones(W.L, bool); mask[idx[bb]] = False
        assert np.array_equal(a[bb, mask], b[bb, mask])
        assert not np.allclose(a[bb, ~mask], b[bb, ~mask])
