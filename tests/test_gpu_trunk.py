"""GPU parity of the dense-sparse-dense trunk (Sec. 3.2 "Three-stage block partition";
Alg. 1): n1 dense blocks, the routed step on n2 blocks, n3 dense blocks, forward and
backward through the C-ABI (paper_2607_02829_amd.trunk) against the oracle's
trunk_forward / trunk_backward on the same seeded inputs.  Indices bit-exact; outputs,
input gradient and every parameter gradient within the normwise bound of the block tests."""
import numpy as np
import pytest

from gpu_helpers import rel_err, tol_for
from oracle import select as osel
from oracle import stack as ostack
from oracle.numerics import storage_to_f64
from paper_2607_02829_amd import device, inputs
from paper_2607_02829_amd.trunk import Trunk

pytestmark = pytest.mark.gpu

CASES = {
    # several tiles and a ragged tail at the small width; the deterministic forecaster's
    # (2, 8, 2) split at the 5.625 deg token count and full width (two samples)
    "small_bf16_121": (inputs.small("trunk_s", Hg=10, Wg=21), (1, 2, 1), 52),
    "small_f32_212": (inputs.small("trunk_f", Hg=9, Wg=11, D=128, H=2, F=512, dtype="f32"), (2, 1, 2), 25),
    "b5625_282": (inputs.WORKLOADS["b5625"].with_(B=2), (2, 8, 2), 128),
}


@pytest.mark.parametrize("case", list(CASES))
def test_trunk_fwd_bwd(case):
    import torch
    w, split, K = CASES[case]
    print(f"[trunk {case}] B={w.B} L={w.L} K={K} D={w.D} split={split} {w.dtype}", flush=True)
    params = inputs.params_to_storage(inputs.block_params(w, sum(split), randomise_affine=True), w.dtype)
    x0 = inputs.to_storage(inputs.token_field(w), w.dtype)
    g3 = inputs.to_storage(inputs.upstream_grad(w), w.dtype)
    seed, step = 11, 3

    tr = Trunk(w, split, params, K=K, seed=seed)
    x0d, g3d = device.to_device(x0), device.to_device(g3)
    x3 = device.to_host(tr.forward(x0d, step))
    g0 = device.to_host(tr.backward(g3d))
    torch.cuda.synchronize()
    got_idx = tr.idx.cpu().numpy()
    grads = [{k: v.cpu().numpy() for k, v in g.items()} for g in tr.block_grads()]
    assert np.array_equal(device.to_host(x0d), x0) and np.array_equal(device.to_host(g3d), g3)

    idx = osel.select_random(w.B, w.L, K, seed, step)
    assert np.array_equal(got_idx, idx)
    print(f"[trunk {case}] oracle", flush=True)
    ref_x3, caches = ostack.trunk_forward(x0, idx, params, split, w.H, 1e-6)
    ref_g0, ref_grads = ostack.trunk_backward(g3, idx, params, split, caches)
    errs = {"x3": rel_err(storage_to_f64(x3), ref_x3), "g0": rel_err(storage_to_f64(g0), ref_g0)}
    for i, (gg, rg) in enumerate(zip(grads, ref_grads)):
        for name in rg:
            if name in ("w_ada", "b_ada"):
                continue
            errs[f"b{i}.{name}"] = rel_err(gg[name], rg[name])
    worst = max(errs, key=errs.get)
    print(f"[trunk {case}] max rel err {errs[worst]:.3e} ({worst})", flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol_for(w.dtype)}
    assert not bad, bad



def test_trunk_bitwise_repeatable():
    # two forward + backward passes of the (2, 8, 2) trunk on the same inputs give identical
    # bits: the three stages share one scratch buffer and each backward's second stream is
    # joined before the next stage runs
    import torch
    w, split, K = CASES["b5625_282"]
    params = inputs.params_to_storage(inputs.block_params(w, sum(split), randomise_affine=True), w.dtype)
    x0 = device.to_device(inputs.to_storage(inputs.token_field(w), w.dtype))
    g3 = device.to_device(inputs.to_storage(inputs.upstream_grad(w), w.dtype))
    tr = Trunk(w, split, params, K=K, seed=4)
    runs = []
    for _ in range(2):
        x3 = tr.forward(x0, 1).clone()
        g0 = tr.backward(g3).clone()
        torch.cuda.synchronize()
        runs.append((x3, g0, [{k: v.clone() for k, v in g.items()} for g in tr.block_grads()]))
    (a3, a0, ag), (b3, b0, bg) = runs
    assert torch.equal(a3.view(torch.int16), b3.view(torch.int16))
    assert torch.equal(a0.view(torch.int16), b0.view(torch.int16))
    for x, y in zip(ag, bg):
        for k in x:
            assert torch.equal(x[k].view(torch.int32), y[k].view(torch.int32)), k


@pytest.mark.parametrize("case,select", [("small_bf16_121", "random"), ("small_f32_212", "random"),
                                         ("b5625_282", "random"), ("b5625_282", "attn")])
def test_trunk_checkpoint_is_bitwise_the_plain_trunk(case, select):
    # activation checkpointing re-runs each stage's forward before its backward from the kept
    # stage input into one shared saved-activation buffer: the deterministic kernels must give
    # the same bits for the output, the input gradient and every parameter gradient, and the
    # forward's output must survive the recompute
    import torch
    w, split, K = CASES[case]
    print(f"[trunk ckpt {case} {select}] B={w.B} L={w.L} K={K} split={split} {w.dtype}", flush=True)
    params = inputs.params_to_storage(inputs.block_params(w, sum(split), randomise_affine=True), w.dtype)
    x0 = device.to_device(inputs.to_storage(inputs.token_field(w), w.dtype))
    g3 = device.to_device(inputs.to_storage(inputs.upstream_grad(w), w.dtype))
    x0_host = device.to_host(x0)
    out = []
    for ck in (False, True):
        tr = Trunk(w, split, params, K=K, seed=5, select=select, checkpoint=ck)
        x3 = tr.forward(x0, 2).clone()
        g0 = tr.backward(g3).clone()
        torch.cuda.synchronize()
        assert torch.equal(tr.x3, x3), "the forward's output changed during the backward"
        out.append((tr.idx.clone(), x3, g0, [{k: v.clone() for k, v in g.items()} for g in tr.block_grads()],
                    tr.saved[0].numel() if ck else sum(s.numel() for s in tr.saved)))
        del tr
    (ia, a3, a0, ag, sa), (ib, b3, b0, bg, sb) = out
    assert np.array_equal(device.to_host(x0), x0_host)
    assert torch.equal(ia, ib)
    bits = torch.int16 if w.dtype == "bf16" else torch.int32
    assert torch.equal(a3.view(bits), b3.view(bits))
    assert torch.equal(a0.view(bits), b0.view(bits))
    for x, y in zip(ag, bg):
        for k in x:
            assert torch.equal(x[k].view(torch.int32), y[k].view(torch.int32)), k
    assert sb < sa, (sb, sa)   # one stage's saved activations instead of all three
    print(f"[trunk ckpt {case} {select}] saved bytes {sa} -> {sb}", flush=True)
