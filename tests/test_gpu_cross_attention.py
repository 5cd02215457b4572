"""GPU parity of the asymmetric attention (Sec. 3.4 "Integration with Generative
Forecasting"): sr_cross_attention_fwd / _bwd with Sq query tokens and Skv key/value tokens
against the oracle's attention forward and backward (fp64) on the same seeded inputs."""
import numpy as np
import pytest

from gpu_helpers import check_pairs, rel_err, tol_for
from oracle import block as oblk
from oracle.numerics import storage_to_f64
from paper_2607_02829_amd import abi, device, inputs

pytestmark = pytest.mark.gpu


def _cfg(B, D, H, dtype):
    return abi.SrConfig(B=B, L=1, D=D, H=H, F=64, n_blocks=1, dtype=abi.SR_BF16 if dtype == "bf16" else abi.SR_F32,
                        kind=abi.SR_BLOCK_PRELN, ln_eps=1e-6, idx_shared=0)


def _data(B, Sq, Skv, D, dtype, seed):
    rng = np.random.default_rng([B, Sq, Skv, D, seed])
    q = inputs.to_storage(rng.standard_normal((B, Sq, D)).astype(np.float32), dtype)
    kv = inputs.to_storage(rng.standard_normal((B, Skv, 2 * D)).astype(np.float32), dtype)
    dO = inputs.to_storage(rng.standard_normal((B, Sq, D)).astype(np.float32), dtype)
    return q, kv, dO


def _gpu(B, Sq, Skv, D, H, dtype, q, kv, dO):
    import torch
    cfg = _cfg(B, D, H, dtype)
    qd, kvd, dOd = device.to_device(q), device.to_device(kv), device.to_device(dO)
    O = torch.empty_like(qd)
    lse = torch.empty((B, H, Sq), dtype=torch.float32, device="cuda")
    abi.sr_cross_attention_fwd(cfg, Sq, Skv, qd, kvd, O, lse)
    dq, dkv = torch.empty_like(qd), torch.empty_like(kvd)
    delta = torch.empty((B, H, Sq), dtype=torch.float32, device="cuda")
    abi.sr_cross_attention_bwd(cfg, Sq, Skv, qd, kvd, O, dOd, lse, dq, dkv, delta)
    torch.cuda.synchronize()
    return device.to_host(O), lse.cpu().numpy(), device.to_host(dq), device.to_host(dkv)


@pytest.mark.parametrize("B,Sq,Skv,D,H,dtype", [
    (2, 37, 130, 256, 4, "bf16"), (2, 130, 37, 256, 4, "bf16"), (1, 1, 50, 128, 4, "f32"),
    (2, 20, 1, 256, 2, "bf16"), (2, 33, 77, 256, 4, "f32"), (1, 64, 200, 256, 8, "bf16"),
    # the MFMA path across its 256-row workgroups and 64-row tiles, ragged on both sides
    (3, 257, 511, 256, 4, "bf16"), (2, 256, 64, 256, 4, "bf16"), (1, 1, 1, 256, 4, "bf16"),
    # head dim 128 (MFMA, 128-row workgroups): ragged on both sides, Sq < Skv and Sq > Skv, one token
    (2, 129, 257, 256, 2, "bf16"), (1, 300, 65, 512, 4, "bf16"), (2, 1, 130, 256, 2, "bf16"),
    (2, 70, 1, 256, 2, "bf16"), (2, 33, 77, 256, 2, "f32"),
])
def test_cross_attention_matches_oracle(B, Sq, Skv, D, H, dtype):
    print(f"[xattn] B={B} Sq={Sq} Skv={Skv} D={D} H={H} {dtype}", flush=True)
    q, kv, dO = _data(B, Sq, Skv, D, dtype, 0)
    O, lse, dq, dkv = _gpu(B, Sq, Skv, D, H, dtype, q, kv, dO)
    q64, kv64, dO64 = storage_to_f64(q), storage_to_f64(kv), storage_to_f64(dO)
    qh = oblk.split_heads(q64, H)
    kh = oblk.split_heads(kv64[..., :D], H)
    vh = oblk.split_heads(kv64[..., D:], H)
    O_ref = oblk.merge_heads(oblk.attention_fwd(qh, kh, vh))
    dq_ref, dk_ref, dv_ref = oblk.attention_bwd(qh, kh, vh, oblk.split_heads(dO64, H))
    tol = tol_for(dtype)
    errs = {"O": rel_err(storage_to_f64(O), O_ref), "dq": rel_err(storage_to_f64(dq), oblk.merge_heads(dq_ref)),
            "dk": rel_err(storage_to_f64(dkv)[..., :D], oblk.merge_heads(dk_ref)),
            "dv": rel_err(storage_to_f64(dkv)[..., D:], oblk.merge_heads(dv_ref))}
    # lse: base-2 log-sum-exp of the scaled scores
    s = np.einsum("bhid,bhjd->bhij", qh, kh) / np.sqrt(D // H)
    lse_ref = (s.max(axis=-1) + np.log(np.exp(s - s.max(axis=-1, keepdims=True)).sum(axis=-1))) / np.log(2.0)
    errs["lse"] = float(np.abs(lse - lse_ref).max() / max(1.0, np.abs(lse_ref).max()))
    print(f"[xattn] errors {errs}", flush=True)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, bad


def test_cross_attention_at_the_generative_shape():
    # 2 samples, 2048 routed queries against all 8192 conditioning tokens, 16 heads, D = 1024:
    # output and every gradient against the fp64 oracle in full
    B, Sq, Skv, D, H = 2, 2048, 8192, 1024, 16
    print(f"[xattn edm] B={B} Sq={Sq} Skv={Skv} D={D} H={H}", flush=True)
    q, kv, dO = _data(B, Sq, Skv, D, "bf16", 1)
    O, lse, dq, dkv = _gpu(B, Sq, Skv, D, H, "bf16", q, kv, dO)
    q64, kv64, dO64 = storage_to_f64(q), storage_to_f64(kv), storage_to_f64(dO)
    qh = oblk.split_heads(q64, H)
    kh = oblk.split_heads(kv64[..., :D], H)
    vh = oblk.split_heads(kv64[..., D:], H)
    print("[xattn edm] oracle", flush=True)
    O_ref = oblk.merge_heads(oblk.attention_fwd(qh, kh, vh))
    dq_ref, dk_ref, dv_ref = oblk.attention_bwd(qh, kh, vh, oblk.split_heads(dO64, H))
    items = [("O", storage_to_f64(O), O_ref), ("dq", storage_to_f64(dq), oblk.merge_heads(dq_ref)),
             ("dk", storage_to_f64(dkv)[..., :D], oblk.merge_heads(dk_ref)),
             ("dv", storage_to_f64(dkv)[..., D:], oblk.merge_heads(dv_ref))]
    check_pairs(items, "bf16", "[xattn edm]")


def test_cross_attention_at_the_generative_shape_hd128():
    # the generative model's heads (8 x 128, App. A.1 EDM table) at 2 x 2048 queries x 8192 keys
    B, Sq, Skv, D, H = 2, 2048, 8192, 1024, 8
    print(f"[xattn edm hd128] B={B} Sq={Sq} Skv={Skv} D={D} H={H}", flush=True)
    q, kv, dO = _data(B, Sq, Skv, D, "bf16", 2)
    O, lse, dq, dkv = _gpu(B, Sq, Skv, D, H, "bf16", q, kv, dO)
    q64, kv64, dO64 = storage_to_f64(q), storage_to_f64(kv), storage_to_f64(dO)
    qh = oblk.split_heads(q64, H)
    kh = oblk.split_heads(kv64[..., :D], H)
    vh = oblk.split_heads(kv64[..., D:], H)
    print("[xattn edm hd128] oracle", flush=True)
    O_ref = oblk.merge_heads(oblk.attention_fwd(qh, kh, vh))
    dq_ref, dk_ref, dv_ref = oblk.attention_bwd(qh, kh, vh, oblk.split_heads(dO64, H))
    items = [("O", storage_to_f64(O), O_ref), ("dq", storage_to_f64(dq), oblk.merge_heads(dq_ref)),
             ("dk", storage_to_f64(dkv)[..., :D], oblk.merge_heads(dk_ref)),
             ("dv", storage_to_f64(dkv)[..., D:], oblk.merge_heads(dv_ref))]
    check_pairs(items, "bf16", "[xattn edm hd128]")


@pytest.mark.parametrize("H", [4, 2])
def test_cross_attention_bitwise_repeatable_hd(H):
    B, Sq, Skv, D = 2, 300, 700, 256
    q, kv, dO = _data(B, Sq, Skv, D, "bf16", 4)
    a = _gpu(B, Sq, Skv, D, H, "bf16", q, kv, dO)
    b = _gpu(B, Sq, Skv, D, H, "bf16", q, kv, dO)
    for x, y in zip(a, b):
        assert np.array_equal(np.ascontiguousarray(x).view(np.uint8), np.ascontiguousarray(y).view(np.uint8))


def test_cross_attention_bitwise_repeatable():
    # deterministic kernels: identical calls give identical bits (forward and backward)
    B, Sq, Skv, D, H = 2, 300, 700, 256, 4
    q, kv, dO = _data(B, Sq, Skv, D, "bf16", 3)
    a = _gpu(B, Sq, Skv, D, H, "bf16", q, kv, dO)
    b = _gpu(B, Sq, Skv, D, H, "bf16", q, kv, dO)
    for x, y in zip(a, b):
        assert np.array_equal(np.ascontiguousarray(x).view(np.uint8), np.ascontiguousarray(y).view(np.uint8))
