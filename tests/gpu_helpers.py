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


def elem_err(a, ref, floor: float = 1e-3) -> float:
    """max_i |a_i - ref_i| / max(|ref_i|, floor * max|ref|): elementwise relative error with a
    floor at 1e-3 of the tensor's largest magnitude."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    big = np.abs(ref).max()
    den = np.maximum(np.abs(ref), floor * (big if big > 0 else 1.0))
    return float((np.abs(a - ref) / den).max())


def row_err(a, ref) -> float:
    """Largest normwise error of one row (last axis): max over rows of
    max|a_row - ref_row| / max|ref_row|.  A wrong row whose values are small against the
    tensor's largest ones still shows here."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.ndim == 1:
        return rel_err(a, ref)
    a2 = a.reshape(-1, ref.shape[-1])
    r2 = ref.reshape(-1, ref.shape[-1])
    den = np.abs(r2).max(axis=1)
    den = np.where(den > 0, den, 1.0)
    return float((np.abs(a2 - r2).max(axis=1) / den).max())


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


def pairs(gpu, ref, kind="preln"):
    """(name, gpu value as fp64, oracle value) for every output and gradient present in both;
    gradients of parameters the block kind does not read must be exactly zero."""
    out = [("h_out", storage_to_f64(gpu["h_out"]), ref["h_out"])]
    if "dh_in" in gpu and "dh_in" in ref:
        out.append(("dh_in", storage_to_f64(gpu["dh_in"]), ref["dh_in"]))
        for i, (gg, rg) in enumerate(zip(gpu["grads"], ref["grads"])):
            for name in gg:
                if kind == "preln" and name in ("w_ada", "b_ada") or kind == "adaln" and name.startswith("ln"):
                    assert not np.any(gg[name]), f"block {i} {name}: unused parameter gradient is not zero"
                    continue
                out.append((f"b{i}.{name}", gg[name], rg[name]))
        if ref.get("dcond") is not None:
            out.append(("dcond", gpu["dcond"], ref["dcond"]))
    return out


def compare(gpu, ref, dtype, kind="preln"):
    """Dict of name -> normwise relative error for every output and gradient present in both."""
    return {n: rel_err(a, r) for n, a, r in pairs(gpu, ref, kind)}


# Tensors whose rows are tokens (outputs and input gradients): each row is held to the bound on
# its own.  Rows of weight gradients are sums over tokens that cancel by construction in places
# (the key rows of dW_qkv: softmax ignores a shift of all keys, so the exact key-bias gradient
# is zero; dW_o, whose bf16 attention outputs share a large component across tokens; dW_ada),
# where the bf16 rounding of the operands is large against the row's own size: their per-row and
# elementwise errors are reported, the bound applies to the whole tensor.
TOKEN_ROWS = ("h_out", "dh_in", "x'", "dx0", "O", "dq", "dk", "dv", "dzc", "dkv")


def check_pairs(items, dtype, label=""):
    """Assert every (name, got, ref) against the stated bound (normwise: max|a - r| / max|r|),
    token tensors also row by row, and print the worst of each measure (normwise, per row,
    elementwise with the 1e-3 floor)."""
    tol = tol_for(dtype)
    norm = {n: rel_err(a, r) for n, a, r in items}
    rows = {n: row_err(a, r) for n, a, r in items}
    elem = {n: elem_err(a, r) for n, a, r in items}
    for d, what in ((norm, "normwise"), (rows, "per-row"), (elem, "elementwise (1e-3 floor)")):
        w = max(d, key=d.get)
        print(f"{label} worst {what}: {d[w]:.3e} ({w})", flush=True)
    tok = {n: rows[n] for n in rows if n.split(".")[-1] in TOKEN_ROWS}
    if tok:
        w = max(tok, key=tok.get)
        print(f"{label} worst per-row of token tensors: {tok[w]:.3e} ({w})", flush=True)
    bad = {n: norm[n] for n in norm if not norm[n] <= tol}
    bad.update({f"{n} (per row)": v for n, v in tok.items() if not v <= tol})
    assert not bad, bad
    return norm, rows, elem
