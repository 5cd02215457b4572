"""Helpers for the GPU parity tests: run the HIP path through the C-ABI binding on
seeded inputs, run the oracle on the same inputs, compare."""
from __future__ import annotations

import numpy as np

from oracle import stack as ostack
from oracle.numerics import storage_to_f64
from paper_2607_02829_amd import abi, device, inputs


def rel_err(a, ref) -> float:
    """max |a - ref| / max |ref| over the tensor (normwise max relative error)."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max()
    return float(np.abs(a - ref).max() / (den if den > 0 else 1.0))


def tol_for(dtype: str) -> float:
    return 2e-2 if dtype == "bf16" else 1e-5


def host_inputs(w, n_blocks=None, randomise_affine=True, S=None, which=0):
    """Seeded storage inputs for a block-stack run on S tokens per sample."""
    S = w.L if S is None else S
    h = inputs.token_field(w, which)[:, :S, :]
    params = inputs.params_to_storage(inputs.block_params(w, n_blocks, randomise_affine=randomise_affine), w.dtype)
    cond = inputs.to_storage(inputs.cond_vector(w), w.dtype) if w.kind == "adaln" else None
    dh = inputs.upstream_grad(w, rows=S)
    return inputs.to_storage(h, w.dtype), params, cond, inputs.to_storage(dh, w.dtype)


def gpu_blocks(w, S, h_st, params, cond, dh_st=None, dense=False):
    """Run sr_sparse_blocks_fwd (and _bwd if dh_st is given) on the GPU."""
    import torch
    nb = len(params)
    cfg = device.config_for(w, n_blocks=nb)
    dp = device.DeviceParams(params, w.kind)
    h_in = device.to_device(h_st)
    h_out = torch.empty_like(h_in)
    c = device.to_device(cond) if cond is not None else None
    saved, scratch = device.workspace(cfg, S)
    if dense:
        abi.sr_dense_blocks_fwd(cfg, dp.array, c, h_in, h_out, saved, scratch)
    else:
        abi.sr_sparse_blocks_fwd(cfg, S, dp.array, c, h_in, h_out, saved, scratch)
    out = {"h_out": device.to_host(h_out)}
    if dh_st is not None:
        g = device.DeviceGrads(w, nb)
        dh = device.to_device(dh_st)
        dh_in = torch.empty_like(dh)
        dcond = torch.empty((w.B, w.D), dtype=torch.float32, device="cuda") if cond is not None else None
        if dense:
            abi.sr_dense_blocks_bwd(cfg, dp.array, c, saved, dh, dh_in, g.array, dcond, scratch)
        else:
            abi.sr_sparse_blocks_bwd(cfg, S, dp.array, c, saved, dh, dh_in, g.array, dcond, scratch)
        torch.cuda.synchronize()
        out["dh_in"] = device.to_host(dh_in)
        out["grads"] = [{k: v.cpu().numpy() for k, v in gg.items()} for gg in g.tensors]
        out["dcond"] = dcond.cpu().numpy() if dcond is not None else None
    torch.cuda.synchronize()
    return out


def oracle_blocks(w, h_st, params, cond, dh_st=None, eps=1e-6):
    p64 = ostack.params_f64(params)
    c64 = storage_to_f64(cond) if cond is not None else None
    h_out, caches = ostack.stack_fwd(storage_to_f64(h_st), p64, w.H, eps, w.kind, c64)
    out = {"h_out": h_out}
    if dh_st is not None:
        dh_in, grads, dcond = ostack.stack_bwd(storage_to_f64(dh_st), p64, caches)
        out.update(dh_in=dh_in, grads=grads, dcond=dcond)
    return out


def compare(gpu, ref, dtype, kind="preln"):
    """Dict of name -> relative error for every output and gradient present in both."""
    errs = {"h_out": rel_err(storage_to_f64(gpu["h_out"]), ref["h_out"])}
    if "dh_in" in gpu and "dh_in" in ref:
        errs["dh_in"] = rel_err(storage_to_f64(gpu["dh_in"]), ref["dh_in"])
        for i, (gg, rg) in enumerate(zip(gpu["grads"], ref["grads"])):
            for name in gg:
                if kind == "preln" and name in ("w_ada", "b_ada") or kind == "adaln" and name.startswith("ln"):
                    assert not np.any(gg[name]), f"block {i} {name}: unused parameter gradient is not zero"
                    continue
                errs[f"b{i}.{name}"] = rel_err(gg[name], rg[name])
        if ref.get("dcond") is not None:
            errs["dcond"] = rel_err(gpu["dcond"], ref["dcond"])
    return errs
