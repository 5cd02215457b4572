#!/usr/bin/env python3
"""Benchmark of the routed middle-block stack on one MI355X.

One step is one pass of the whole hot path over one batch:
    select -> gather -> blocks fwd -> residual-delta scatter
           -> gather(g) -> blocks bwd -> scatter(g)
(Alg. 1 stage 2 and its backward; by default through the fused calls, which gather into
the stack's first step and scatter from its last; --unfused times the separate calls),
on the 0.25 deg workload by default:
B=1, 90 x 180 token grid (L=16200), keep 25% (K=4050), D=1024, 16 heads, MLP 4096,
12 middle blocks, bf16 storage with fp32 accumulation, synthetic smooth token
fields and N(0, 0.02) weights, all resident in HBM before timing starts.

Prints ONE JSON line: routed tokens/s (B*K per step time), ms/step, the
dense keep=100% step time and speedup, peak memory of both modes, the roofline
of the dominant kernel (HIP-event timing inside the timed region), and the CPU
oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_FLOPS = 2.5e15      # MI355X dense bf16 MFMA
PEAK_HBM_BYTES = 8.0e12       # MI355X HBM3E
COPY_PROBE_BYTES = 1 << 30    # device-to-device copy of known size (counter calibration)
PROFILES = os.path.join(ROOT, "profiles")

# kernel group -> (source file whose text the HBM-traffic figure was taken on, kernel symbol)
KERNEL_SOURCES = {
    "attn_bwd_dkv": ("paper_2607_02829_amd/csrc/attention.hip", "attn_bwd_dkv_mfma"),
    "attn_bwd_dq": ("paper_2607_02829_amd/csrc/attention.hip", "attn_bwd_dq_mfma"),
    "attn_fwd": ("paper_2607_02829_amd/csrc/attention.hip", "attn_fwd_mfma"),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Step:
    """Device buffers and the launch sequence of one routed (or dense) step."""

    def __init__(self, w, dense: bool, seed: int = 42, fused: bool = True):
        import torch
        from paper_2607_02829_amd import abi, device, inputs
        self.abi, self.w, self.dense, self.fused = abi, w, dense, fused
        self.cfg = device.config_for(w)
        self.K = w.L if dense else w.K
        self.S = self.K
        self.seed = seed
        x = inputs.to_storage(inputs.token_field(w, 0), w.dtype)
        self.x = device.to_device(x)
        self.g = device.to_device(inputs.to_storage(inputs.upstream_grad(w), w.dtype))
        self.params = device.DeviceParams(inputs.params_to_storage(inputs.block_params(w), w.dtype), w.kind)
        self.cond = device.to_device(inputs.to_storage(inputs.cond_vector(w), w.dtype)) if w.kind == "adaln" else None
        self.dcond = torch.empty((w.B, w.D), dtype=torch.float32, device="cuda") if w.kind == "adaln" else None
        self.grads = device.DeviceGrads(w, w.n_blocks, skip_unused=True)
        self.saved, self.scratch = device.workspace(self.cfg, self.S)
        self.sel = abi.SR_SEL_TOPK_DIFFNORM if w.select == "topk" else abi.SR_SEL_RANDOM
        if self.sel == abi.SR_SEL_TOPK_DIFFNORM:
            self.x_prev = device.to_device(inputs.to_storage(inputs.token_field(w, 1), w.dtype))
            self.sel_scratch = torch.empty(abi.sr_select_scratch_bytes(self.cfg, self.sel), dtype=torch.uint8,
                                           device="cuda")
        else:
            self.x_prev = self.sel_scratch = None
        if not dense:
            self.idx = torch.empty((w.B, self.K), dtype=torch.int32, device="cuda")
            self.h0 = torch.empty((w.B, self.K, w.D), dtype=self.x.dtype, device="cuda")
            self.h = torch.empty_like(self.h0)
            self.gh = torch.empty_like(self.h0)
            self.dh = torch.empty_like(self.h0)
        else:
            self.x_out = torch.empty_like(self.x)
            self.dx = torch.empty_like(self.x)

    def run(self, step: int):
        a, c, K, S = self.abi, self.cfg, self.K, self.S
        p, g = self.params.array, self.grads.array
        if self.dense:
            a.sr_dense_blocks_fwd(c, p, self.cond, self.x, self.x_out, self.saved, self.scratch)
            a.sr_dense_blocks_bwd(c, p, self.cond, self.saved, self.g, self.dx, g, self.dcond, self.scratch)
            return
        x_t = self.x if self.sel == a.SR_SEL_TOPK_DIFFNORM else None
        a.sr_select_indices(c, K, self.sel, self.seed, step, x_t, self.x_prev, self.idx, self.sel_scratch)
        if self.fused:   # gather and scatter fused into the stack's first and last steps
            a.sr_routed_blocks_fwd(c, K, self.idx, p, self.cond, self.x, self.saved)
            a.sr_routed_blocks_bwd(c, K, self.idx, p, self.cond, self.saved, self.g, g, self.dcond, self.scratch)
            return
        a.sr_gather(c, K, self.x, self.idx, self.h0)
        a.sr_sparse_blocks_fwd(c, S, p, self.cond, self.h0, self.h, self.saved, self.scratch)
        a.sr_scatter_delta(c, K, self.x, self.h, self.h0, self.idx)
        a.sr_gather(c, K, self.g, self.idx, self.gh)
        a.sr_sparse_blocks_bwd(c, S, p, self.cond, self.saved, self.gh, self.dh, g, self.dcond, self.scratch)
        a.sr_scatter_delta(c, K, self.g, self.dh, None, self.idx)


def time_steps(st: Step, steps: int, warmup: int, start: int = 0, profile_filter: str | None = None):
    import torch
    for i in range(warmup):
        st.run(start + i)
    torch.cuda.synchronize()
    prof = None
    if profile_filter is not None:
        st.abi.sr_profile_start(profile_filter)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for i in range(steps):
        st.run(start + warmup + i)
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    if profile_filter is not None:
        prof = st.abi.sr_profile_stop()
    return (t1 - t0) * 1e3 / steps, ev0.elapsed_time(ev1) / steps, prof


class TrunkStep:
    """The whole trunk with a (2, n - 4, 2) dense-sparse-dense split (the deterministic
    forecaster's (2, 8, 2) at 12 blocks): forward + backward of all n blocks per step."""

    def __init__(self, w, seed: int = 42, split=None, K: int | None = None, select: str = "random",
                 checkpoint: bool = False):
        from paper_2607_02829_amd import device, inputs
        from paper_2607_02829_amd.trunk import Trunk
        self.split = (2, w.n_blocks - 4, 2) if split is None else tuple(split)
        params = inputs.params_to_storage(inputs.block_params(w, sum(self.split)), w.dtype)
        self.trunk = Trunk(w, self.split, params, K=K, seed=seed, select=select, checkpoint=checkpoint)
        self.x0 = device.to_device(inputs.to_storage(inputs.token_field(w, 0), w.dtype))
        self.g3 = device.to_device(inputs.to_storage(inputs.upstream_grad(w), w.dtype))

    def run(self, step: int):
        self.trunk.forward(self.x0, step)
        self.trunk.backward(self.g3)


def block_flops(w, S: int, n_blocks: int | None = None) -> float:
    """Algorithmic FLOPs of the pre-LN / adaLN blocks' forward + backward on S tokens per sample
    (3 x the forward's M (24 D^2 + 4 S D) at F = 4D; no attention recompute counted)."""
    nb = w.n_blocks if n_blocks is None else n_blocks
    M = w.B * S
    return 3.0 * nb * (2 * M * (3 * w.D * w.D + w.D * w.D + 2 * w.D * w.F) + 4.0 * w.B * S * S * w.D)


def workload_summary(name: str, steps: int = 5, dense_steps: int = 2) -> dict:
    """Routed and dense step of another workload (fused routed calls as in the main line):
    ms per step, routed tokens/s, speedup over dense, and the stack's MFMA fraction."""
    import torch
    from paper_2607_02829_amd import inputs
    w = inputs.WORKLOADS[name]
    sp = Step(w, dense=False)
    sp.run(0)
    torch.cuda.synchronize()
    ms, _, _ = time_steps(sp, steps, 2, start=1)
    del sp
    torch.cuda.empty_cache()
    dn = Step(w, dense=True)
    dn.run(0)
    torch.cuda.synchronize()
    dms, _, _ = time_steps(dn, dense_steps, 1, start=1)
    del dn
    torch.cuda.empty_cache()
    rec = {"config": f"B={w.B}, {w.Hg}x{w.Wg} tokens (L={w.L}), K={w.K}, D={w.D}, H={w.H}, F={w.F}, "
                     f"{w.n_blocks} {w.kind} blocks, {w.select} selection, {w.dtype}",
           "ms_per_step": round(ms, 3), "routed_tokens_per_s": round(w.B * w.K / (ms * 1e-3), 1),
           "dense_ms_per_step": round(dms, 3), "speedup_vs_dense": round(dms / ms, 3),
           "stack_mfma_frac": round(block_flops(w, w.K) / (ms * 1e-3) / PEAK_BF16_FLOPS, 4),
           "dense_stack_mfma_frac": round(block_flops(w, w.L) / (dms * 1e-3) / PEAK_BF16_FLOPS, 4)}
    log(f"workload {name}: {ms:.2f} ms routed, {dms:.2f} ms dense, speedup {rec['speedup_vs_dense']}")
    return rec


class GenStep:
    """The generative model's sparse middle stage (Alg. 2 stage 2): select K tokens of Z_x, gather,
    the blocks (FiLM, self-attention on the K tokens, sigma-gated cross-attention to all L
    conditioning tokens, MLP), residual-delta scatter, and the backward through the same routing;
    or (dense) the same blocks on all L tokens of Z_x."""

    def __init__(self, w, dense: bool, seed: int = 42):
        import torch
        from paper_2607_02829_amd import abi, device, inputs
        self.abi, self.w, self.dense, self.seed = abi, w, dense, seed
        self.cfg = abi.SrConfig(B=w.B, L=w.L, D=w.D, H=w.H, F=w.F, n_blocks=w.n_blocks, dtype=abi.SR_BF16,
                                kind=abi.SR_BLOCK_PRELN, ln_eps=1e-6, idx_shared=0)
        self.K = w.L if dense else w.K
        st = lambda a: device.to_device(inputs.to_storage(a, w.dtype))
        self.x, self.zc, self.e = st(inputs.token_field(w, 0)), st(inputs.conditioning_tokens(w)), \
            st(inputs.noise_embedding(w))
        self.g = st(inputs.upstream_grad(w))
        self.params = device.DeviceEdmParams(inputs.params_to_storage(inputs.edm_block_params(w), w.dtype))
        self.grads = device.DeviceEdmGrads(w.D, w.F, w.n_blocks)
        self.dzc = torch.empty((w.B, w.L, w.D), dtype=torch.float32, device="cuda")
        self.de = torch.empty((w.B, w.D), dtype=torch.float32, device="cuda")
        self.saved, self.scratch = device.edm_workspace(self.cfg, self.K)
        if dense:
            self.x_out, self.dx = torch.empty_like(self.x), torch.empty_like(self.x)
        else:
            self.idx = torch.empty((w.B, self.K), dtype=torch.int32, device="cuda")
            self.h0 = torch.empty((w.B, self.K, w.D), dtype=self.x.dtype, device="cuda")
            self.h, self.gh, self.dh = torch.empty_like(self.h0), torch.empty_like(self.h0), torch.empty_like(self.h0)

    def run(self, step: int):
        a, c, K, p, g = self.abi, self.cfg, self.K, self.params.array, self.grads.array
        if self.dense:
            a.sr_edm_blocks_fwd(c, K, p, self.e, self.zc, self.x, self.x_out, self.saved)
            a.sr_edm_blocks_bwd(c, K, p, self.e, self.zc, self.saved, self.g, self.dx, g, self.dzc, self.de,
                                self.scratch)
            return
        a.sr_select_indices(c, K, a.SR_SEL_RANDOM, self.seed, step, None, None, self.idx)
        a.sr_gather(c, K, self.x, self.idx, self.h0)
        a.sr_edm_blocks_fwd(c, K, p, self.e, self.zc, self.h0, self.h, self.saved)
        a.sr_scatter_delta(c, K, self.x, self.h, self.h0, self.idx)
        a.sr_gather(c, K, self.g, self.idx, self.gh)
        a.sr_edm_blocks_bwd(c, K, p, self.e, self.zc, self.saved, self.gh, self.dh, g, self.dzc, self.de,
                            self.scratch)
        a.sr_scatter_delta(c, K, self.g, self.dh, None, self.idx)


def edm_flops(w, S: int) -> float:
    """Algorithmic FLOPs of the generative blocks' forward + backward on S query tokens with L
    conditioning tokens: the S-row GEMMs (QKV, O, Q, O_c, FC1, FC2), the K/V projection of the L
    conditioning rows, self-attention over S and cross-attention S x L; 3 x the forward."""
    D, F = w.D, w.F
    M, Mc = w.B * S, w.B * w.L
    fwd = 2.0 * M * (3 * D * D + 3 * D * D + 2 * D * F) + 2.0 * Mc * 2 * D * D \
        + 4.0 * w.B * S * S * D + 4.0 * w.B * S * w.L * D
    return 3.0 * w.n_blocks * fwd


def generative_stage(steps: int = 5, dense_steps: int = 3) -> dict:
    """The generative model's sparse middle stage against its dense blocks at the 1.40625 deg token
    grid (B = 2, L = 8192, K = 2048, D = 1024, 8 heads of 128, F = 4096, the 4 middle blocks of the
    (2, 4, 2) split): ms per fwd + bwd step, speedup, MFMA fraction, peak memory."""
    import torch
    from paper_2607_02829_amd import inputs
    w = inputs.WORKLOADS["gen"]
    out = {"config": f"B={w.B}, {w.Hg}x{w.Wg} tokens (L={w.L}), K={w.K}, D={w.D}, {w.H} heads of {w.hd}, F={w.F}, "
                     f"{w.n_blocks} generative blocks (FiLM, self-attention, sigma-gated cross-attention to all "
                     f"L conditioning tokens, MLP), random selection, bf16"}
    for dense in (False, True):
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        st = GenStep(w, dense)
        st.run(0)
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - base
        ms, _, _ = time_steps(st, dense_steps if dense else steps, 1, start=1)
        finite = bool(torch.isfinite((st.dx if dense else st.g).float()).all().item())
        del st
        torch.cuda.empty_cache()
        S = w.L if dense else w.K
        out["dense" if dense else "sparse"] = {
            "ms_per_step": round(ms, 3), "peak_bytes": int(peak),
            "mfma_frac": round(edm_flops(w, S) / (ms * 1e-3) / PEAK_BF16_FLOPS, 4), "outputs_finite": finite}
    out["routed_tokens_per_s"] = round(w.B * w.K / (out["sparse"]["ms_per_step"] * 1e-3), 1)
    out["speedup_vs_dense"] = round(out["dense"]["ms_per_step"] / out["sparse"]["ms_per_step"], 3)
    out["peak_ratio"] = round(out["dense"]["peak_bytes"] / out["sparse"]["peak_bytes"], 3)
    log(f"generative stage: {out['sparse']['ms_per_step']} ms sparse, {out['dense']['ms_per_step']} ms dense, "
        f"speedup {out['speedup_vs_dense']}")
    return out


def trunk_sweep(w, dense_ms: float | None, steps: int = 3) -> dict:
    """The trunk over the keep ratios of the paper's keep-ratio ablation at the (2, n-4, 2)
    split, and over the block splits of its split ablation at r = 0.25 (Sec. 4.4, "Effect of
    keep ratio" / "Effect of block split"): ms per fwd + bwd step and speedup over the dense
    n-block step.  K = floor(r L) per sample; r = 1 routes every token through the middle."""
    import math
    import torch
    from paper_2607_02829_amd.trunk import eq_speedup_estimate
    out = {"keep": [], "split": []}
    n = w.n_blocks
    runs = [("keep", (2, n - 4, 2), r) for r in (0.10, 0.25, 0.50, 0.75, 1.0)]
    runs += [("split", s, 0.25) for s in ((1, n - 2, 1), (3, n - 6, 3), (4, n - 8, 4)) if min(s) >= 1]
    for kind, split, r in runs:
        K = max(1, math.floor(r * w.L))
        tr = TrunkStep(w, split=split, K=K)
        tr.run(0)
        torch.cuda.synchronize()
        tms, _, _ = time_steps(tr, steps, 1, start=1)
        n1, n2, n3 = split
        rec = {"split": list(split), "keep": r, "K": K, "ms_per_step": round(tms, 3),
               "speedup_vs_dense": round(dense_ms / tms, 3) if dense_ms else None,
               "eq_speedup_estimate": round(eq_speedup_estimate(split, r), 3)}
        out[kind].append(rec)
        log(f"trunk {kind}: split {split} r={r} K={K}: {tms:.2f} ms, speedup {rec['speedup_vs_dense']}")
        del tr
        torch.cuda.empty_cache()
    return out


def graph_timing(st: Step, steps: int, warmup: int) -> dict:
    """Capture one routed step (selection + the fused forward and backward, whose second-stream
    weight gradients are forked and joined inside the capture) in a HIP graph and time its
    replays: the launch cost of ~40 kernels per block leaves the step.  Every replay redoes the
    whole step on the current state, with the draw fixed at capture (a graph replays its launch
    arguments)."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        st.run(10_000)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st.run(10_001)
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    finite = bool(torch.isfinite(st.x.float()).all().item() and torch.isfinite(st.g.float()).all().item())
    del g
    return {"ms_per_step": round(ms, 4), "routed_tokens_per_s": round(st.w.B * st.K / (ms * 1e-3), 1),
            "outputs_finite": finite}


def cross_attention_timing(reps: int = 5) -> dict:
    """The asymmetric attention of the generative block's sparse stage at its shape (2 samples,
    2048 routed queries against 8192 conditioning tokens, D = 1024, bf16) with 16 heads of 64 and
    with the generative model's 8 heads of 128."""
    return {f"heads_{H}x{1024 // H}": cross_attention_one(H, reps) for H in (16, 8)}


def cross_attention_one(H: int, reps: int = 5) -> dict:
    """Forward and backward through sr_cross_attention_fwd / _bwd (the MFMA attention kernels),
    HIP-event timed; algorithmic FLOPs 4 B Sq Skv D forward, 8 B Sq Skv D backward."""
    import torch
    from paper_2607_02829_amd import abi
    B, Sq, Skv, D = 2, 2048, 8192, 1024
    cfg = abi.SrConfig(B=B, L=1, D=D, H=H, F=64, n_blocks=1, dtype=abi.SR_BF16, kind=abi.SR_BLOCK_PRELN,
                       ln_eps=1e-6, idx_shared=0)
    g = torch.Generator(device="cuda").manual_seed(5)
    q = torch.randn((B, Sq, D), device="cuda", generator=g).to(torch.bfloat16)
    kv = torch.randn((B, Skv, 2 * D), device="cuda", generator=g).to(torch.bfloat16)
    dO = torch.randn((B, Sq, D), device="cuda", generator=g).to(torch.bfloat16)
    O, dq, dkv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(kv)
    lse = torch.empty((B, H, Sq), dtype=torch.float32, device="cuda")
    delta = torch.empty_like(lse)
    times = {"fwd": [], "bwd": []}
    for r in range(reps + 1):
        for name in ("fwd", "bwd"):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            if name == "fwd":
                abi.sr_cross_attention_fwd(cfg, Sq, Skv, q, kv, O, lse)
            else:
                abi.sr_cross_attention_bwd(cfg, Sq, Skv, q, kv, O, dO, lse, dq, dkv, delta)
            e1.record()
            torch.cuda.synchronize()
            if r > 0:
                times[name].append(e0.elapsed_time(e1))
    out = {"shape": {"B": B, "Sq": Sq, "Skv": Skv, "D": D, "H": H}, "kernels": f"mfma (bf16, head dim {D // H})"}
    for name, mult in (("fwd", 4.0), ("bwd", 8.0)):
        ms = sorted(times[name])[len(times[name]) // 2]
        flops = mult * B * Sq * Skv * D
        out[name] = {"ms": round(ms, 3), "TFLOP/s": round(flops / (ms * 1e-3) / 1e12, 1),
                     "frac_of_2.5PF": round(flops / (ms * 1e-3) / PEAK_BF16_FLOPS, 4)}
    return out


def kernel_breakdown(st: Step, step_index: int):
    """One profiled step with every launch group bracketed by events."""
    import torch
    torch.cuda.synchronize()
    st.abi.sr_profile_start("")
    st.run(step_index)
    torch.cuda.synchronize()
    return st.abi.sr_profile_stop()


def source_hash(group: str) -> str | None:
    import hashlib
    if group not in KERNEL_SOURCES:
        return None
    with open(os.path.join(ROOT, KERNEL_SOURCES[group][0]), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_for(group: str, workload: str):
    """HBM bytes per launch from the committed counter summary, if it was taken on the
    current source of the kernel (else None)."""
    path = os.path.join(PROFILES, f"{group}_{workload}_hbm_traffic.md")
    if not os.path.exists(path) or source_hash(group) is None:
        return None
    fields = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            fields[k.strip()] = v.strip().strip("`")
    if fields.get("source_sha256") != source_hash(group):
        return None
    return float(fields["hbm_bytes_per_launch"])


def summarize_pmc(group: str, workload: str, fetch_csv: str, write_csv: str, command: str) -> str:
    """Turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE; KiB per dispatch) into the
    per-launch HBM traffic of `group`, scaled by the counters of the copy probe."""
    import csv
    import statistics

    def per_kernel(path, counter):
        vals = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return vals

    sym = KERNEL_SOURCES[group][1]
    fetch, write = per_kernel(fetch_csv, "FETCH_SIZE"), per_kernel(write_csv, "WRITE_SIZE")

    def pick(vals, needle):
        keys = [k for k in vals if needle in k]
        if not keys:
            raise SystemExit(f"no dispatch of {needle} in the counter file")
        return statistics.mean(vals[keys[0]]), len(vals[keys[0]]), keys[0]

    def copy_entry(vals):
        # the copy probe is the largest dispatch of the runtime's buffer-copy kernel (torch's
        # elementwise "copy" kernels convert types and read a different number of bytes)
        best = None
        for k, v in vals.items():
            if "copyBuffer" in k:
                m = max(v)
                if best is None or m > best[0]:
                    best = (m, k)
        if best is None:
            raise SystemExit("no copy-probe dispatch in the counter file")
        return best

    f_k, n_k, name = pick(fetch, sym)
    w_k, _, _ = pick(write, sym)
    f_c, copy_name = copy_entry(fetch)
    w_c, _ = copy_entry(write)
    f_scale = COPY_PROBE_BYTES / (f_c * 1024.0)
    w_scale = COPY_PROBE_BYTES / (w_c * 1024.0)
    total = f_k * 1024.0 * f_scale + w_k * 1024.0 * w_scale
    lines = [
        f"# HBM traffic of `{sym}` on the {workload} workload",
        "",
        "rocprofv3 counter passes (one counter group per run), KiB per dispatch, averaged over",
        f"{n_k} dispatches of the kernel; scaled by the same counters read on a device-to-device",
        f"copy of {COPY_PROBE_BYTES} bytes (`{copy_name.split('(')[0]}`).",
        "",
        "Commands (repository root on the MI355X machine, `cd /tmp && export TMPDIR=/tmp` first):",
        "",
        "```",
        command,
        "```",
        "",
        f"- kernel: `{name.split('(')[0]}`",
        f"- fetch_kib_per_launch: {f_k:.1f}",
        f"- write_kib_per_launch: {w_k:.1f}",
        f"- copy_probe_fetch_kib: {f_c:.1f}",
        f"- copy_probe_write_kib: {w_c:.1f}",
        f"- fetch_scale: {f_scale:.4f}",
        f"- write_scale: {w_scale:.4f}",
        f"- hbm_bytes_per_launch: {total:.0f}",
        f"- source_sha256: `{source_hash(group)}`",
        "",
    ]
    return "\n".join(lines)


# routing kernels: symbol -> (label, algorithmic bytes of one dispatch on `rows` rows of D columns)
# kernel symbol: (what it does, algorithmic bytes for `rows` routed rows of D columns)
ROUTING_KERNELS = {
    "gather_kernel": ("gather (h0 = x[idx], bf16)", lambda rows, D: 2 * rows * D * 2 + 4 * rows),
    "scatter_delta_kernel": ("residual-delta scatter, h0 re-read from x (bf16)", lambda rows, D: 3 * rows * D * 2 + 4 * rows),
    "gather_rows_f32_kernel": ("gradient gather into fp32 + bf16 copies (backward)", lambda rows, D: rows * D * 8 + 4 * rows),
    "scatter_f32_delta_kernel": ("rounding + residual-delta scatter of the fp32 gradient (backward)",
                                 lambda rows, D: rows * D * 8 + 4 * rows),
    "ln_fwd_kernel": ("first LayerNorm with the gather (forward): x[idx] -> fp32 copy + LN1",
                      lambda rows, D: rows * D * 8 + 12 * rows),
}
ROUTING_ROWS_PER_BLOCK = 4   # one wave per row, four waves per 256-thread workgroup
ROUTING_ROWS_PER_WAVE = {"gather_kernel": 2}   # the others take one row per wave


def summarize_routing_pmc(fetch_csv: str, write_csv: str, command: str, D: int = 1024) -> str:
    """HBM traffic of the routing kernels per dispatch size from two rocprofv3 --pmc runs
    (FETCH_SIZE, WRITE_SIZE), scaled by the copy probe, against their algorithmic bytes."""
    import csv
    import statistics

    def per_dispatch(path, counter):
        out = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            out.setdefault((r["Kernel_Name"], int(r["Grid_Size"])), []).append(float(r["Counter_Value"]))
        return out

    fetch, write = per_dispatch(fetch_csv, "FETCH_SIZE"), per_dispatch(write_csv, "WRITE_SIZE")
    copy = [(max(v), k) for k, v in fetch.items() if "copyBuffer" in k[0]]
    copyw = [(max(v), k) for k, v in write.items() if "copyBuffer" in k[0]]
    if not copy or not copyw:
        raise SystemExit("no copy-probe dispatch in the counter files")
    f_scale = COPY_PROBE_BYTES / (max(copy)[0] * 1024.0)
    w_scale = COPY_PROBE_BYTES / (max(copyw)[0] * 1024.0)
    lines = [
        "# HBM traffic of the routing kernels (gather, residual-delta scatter and their fused forms)",
        "",
        "rocprofv3 counter passes (one counter per run), KiB per dispatch averaged over the dispatches",
        f"of one kernel and grid size, scaled by the same counters on a {COPY_PROBE_BYTES}-byte device copy",
        f"(FETCH_SIZE x {f_scale:.4f}, WRITE_SIZE x {w_scale:.4f}); rows = grid threads / 64 x rows per wave",
        "(two for the gather, one for the others; the grid's last workgroup may be partly idle);",
        "algorithmic bytes as in `bench.py` (one read of each input, one write of each output).",
        "",
        "Commands (repository root on the MI355X machine, `cd /tmp && export TMPDIR=/tmp` first):",
        "",
        "```",
        command,
        "```",
        "",
        "| kernel | rows | dispatches | fetch MB | write MB | HBM MB | algorithmic MB | HBM / algorithmic |",
        "|---|---:|---:|---:|---:|---:|---:|---:|",
    ]
    for (name, grid), fv in sorted(fetch.items(), key=lambda kv: (kv[0][0], kv[0][1])):
        sym = next((k for k in ROUTING_KERNELS if k in name.split("(")[0]), None)
        if sym is None or (name, grid) not in write:
            continue
        if sym == "ln_fwd_kernel":   # only the gathering form (fifth template argument)
            targs = name.split("(")[0].split("<", 1)[-1].rstrip(">").split(", ")
            if len(targs) < 5 or targs[4] != "true":
                continue
        rows = grid // 64 * ROUTING_ROWS_PER_WAVE.get(sym, 1)
        f = statistics.mean(fv) * 1024.0 * f_scale
        w = statistics.mean(write[(name, grid)]) * 1024.0 * w_scale
        alg = ROUTING_KERNELS[sym][1](rows, D)
        lines.append(f"| `{sym}` ({ROUTING_KERNELS[sym][0]}) | {rows} | {len(fv)} | {f / 1e6:.2f} | {w / 1e6:.2f} | "
                     f"{(f + w) / 1e6:.2f} | {alg / 1e6:.2f} | {(f + w) / alg:.3f} |")
    lines.append("")
    return "\n".join(lines)


def routing_sweep(D: int, sizes=(4050, 32768, 262144), reps: int = 5) -> list:
    """HBM bandwidth of the gather and the residual-delta scatter (bf16, D columns, h0 read from x)
    on one sample of L = 2K tokens, for K routed rows per call; a 512 MB write between calls
    evicts the Infinity Cache, so the large sizes measure HBM.  Algorithmic bytes: gather
    2KD*2 + 4K, scatter 3KD*2 + 4K."""
    import torch
    from paper_2607_02829_amd import abi
    evict = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    out = []
    for K in sizes:
        L = 2 * K
        cfg = abi.SrConfig(B=1, L=L, D=D, H=max(1, D // 64), F=4 * D, n_blocks=1, dtype=abi.SR_BF16,
                           kind=abi.SR_BLOCK_PRELN, ln_eps=1e-6, idx_shared=0)
        x = torch.randn((1, L, D), device="cuda").to(torch.bfloat16)
        idx = torch.empty((1, K), dtype=torch.int32, device="cuda")
        abi.sr_select_indices(cfg, K, abi.SR_SEL_RANDOM, 7, 0, None, None, idx)
        h0 = torch.empty((1, K, D), dtype=torch.bfloat16, device="cuda")
        h = torch.empty_like(h0)
        times = {"gather": [], "scatter_delta": []}
        for r in range(reps + 1):
            for name in ("gather", "scatter_delta"):
                evict.zero_()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                if name == "gather":
                    abi.sr_gather(cfg, K, x, idx, h0)
                else:   # h0 = NULL: the gathered rows are re-read from x (the backward's form)
                    abi.sr_scatter_delta(cfg, K, x, h, None, idx)
                e1.record()
                torch.cuda.synchronize()
                if r > 0:
                    times[name].append(e0.elapsed_time(e1))
        for name, nbytes in (("gather", 2 * K * D * 2 + 4 * K), ("scatter_delta", 3 * K * D * 2 + 4 * K)):
            ms = sorted(times[name])[len(times[name]) // 2]
            gbs = nbytes / (ms * 1e-3) / 1e9
            out.append({"kernel": name, "rows": K, "bytes": nbytes, "us": round(ms * 1e3, 2),
                        "GB/s": round(gbs, 1), "frac_of_8TB/s": round(gbs * 1e9 / PEAK_HBM_BYTES, 3)})
        del x, idx, h0, h
    # reference: a plain device-to-device copy of the largest gather's size (reads and writes
    # the same bytes contiguously), timed the same way
    n = 2 * sizes[-1] * D * 2
    src = torch.empty(n // 2, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    times = []
    for r in range(reps + 1):
        evict.zero_()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        if r > 0:
            times.append(e0.elapsed_time(e1))
    ms = sorted(times)[len(times) // 2]
    gbs = n / (ms * 1e-3) / 1e9
    out.append({"kernel": "device copy (reference)", "rows": sizes[-1], "bytes": n, "us": round(ms * 1e3, 2),
                "GB/s": round(gbs, 1), "frac_of_8TB/s": round(gbs * 1e9 / PEAK_HBM_BYTES, 3)})
    del src, dst, evict
    torch.cuda.empty_cache()
    return out


def cpu_baseline(w, n_sample: int = 3) -> dict:
    """Time the oracle on a bounded sample: n_sample blocks forward+backward on the K routed
    tokens of one sample (about 10 s of CPU work at the 0.25 deg shape) plus the routing
    (selection, gather, scatter) of one step; the step time is estimated as
    n_blocks / n_sample x the sampled blocks + routing."""
    import numpy as np
    from oracle import routing as orouting
    from oracle import select as osel
    from oracle import stack as ostack
    from oracle.numerics import storage_to_f64
    from paper_2607_02829_amd import inputs

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # noqa: BLE001
        cores = os.cpu_count() or 1
    K = w.K
    n_sample = max(1, min(n_sample, w.n_blocks))
    x = inputs.to_storage(inputs.token_field(w), w.dtype)[:1]
    p = ostack.params_f64(inputs.params_to_storage(inputs.block_params(w, n_sample), w.dtype))
    t0 = time.perf_counter()
    idx = osel.select_random(1, w.L, K, 42, 0)
    h0 = orouting.gather(x, idx)
    t1 = time.perf_counter()
    out, caches = ostack.stack_fwd(storage_to_f64(h0), p, w.H, 1e-6, w.kind)
    ostack.stack_bwd(np.ones_like(out), p, caches)
    t3 = time.perf_counter()
    orouting.scatter_delta(x, h0, h0, idx)
    t4 = time.perf_counter()
    routing_s = (t1 - t0) + (t4 - t3)
    blocks_s = t3 - t1
    step_s = w.B * (w.n_blocks / n_sample * blocks_s + 2 * routing_s)
    return {"value": w.B * K / step_s, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"fp64 oracle: {n_sample} blocks fwd+bwd on {K} routed tokens of 1 sample ({blocks_s:.1f} s) "
                       f"plus select/gather/scatter ({routing_s:.2f} s); step = B x (n_blocks / {n_sample} x "
                       f"sampled blocks + 2 x routing) = {step_s:.1f} s (extrapolated)")}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="d025", help="tiny | b5625 | c1406 | d025 | edm")
    ap.add_argument("--dense-steps", type=int, default=3, help="timed steps of the dense keep=100%% mode (0: skip)")
    ap.add_argument("--trunk-steps", type=int, default=3,
                    help="timed steps of the whole (2, n-4, 2) trunk, pre-LN workloads (0: skip)")
    ap.add_argument("--no-trunk-sweep", action="store_true",
                    help="skip the trunk over keep ratios 0.10-1.0 and block splits (pre-LN workloads)")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the routed and dense steps of the other grids (5.625, 1.40625 deg, diffusion)")
    ap.add_argument("--no-generative", action="store_true",
                    help="skip the generative model's sparse middle stage against its dense blocks")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-routing-sweep", action="store_true", help="skip the gather/scatter bandwidth sweep")
    ap.add_argument("--breakdown", action="store_true", help="print the per-kernel breakdown to stderr")
    ap.add_argument("--graph", action="store_true",
                    help="also time the fused routed step captured once in a HIP graph and replayed (the draw is "
                         "the one fixed at capture)")
    ap.add_argument("--cross-attention", action="store_true",
                    help="also time the generative block's asymmetric attention (2048 queries x 8192 keys)")
    ap.add_argument("--unfused", action="store_true",
                    help="time the routed step as separate gather / blocks / scatter calls (default: the fused "
                         "sr_routed_blocks_fwd/bwd)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run one device-to-device copy of known size first (counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("GROUP", "FETCH_CSV", "WRITE_CSV", "OUT_MD"),
                    help="write the HBM-traffic summary of GROUP from two rocprofv3 --pmc CSVs and exit")
    ap.add_argument("--pmc-command", default="", help="command text recorded in the summary")
    ap.add_argument("--summarize-routing-pmc", nargs=3, metavar=("FETCH_CSV", "WRITE_CSV", "OUT_MD"),
                    help="write the routing kernels' HBM-traffic summary from two rocprofv3 --pmc CSVs and exit")
    ap.add_argument("--generative-only", action="store_true",
                    help="time only the generative stage against its dense blocks (one JSON line)")
    args = ap.parse_args()

    if args.summarize_pmc:
        group, fcsv, wcsv, out_md = args.summarize_pmc
        text = summarize_pmc(group, args.workload, fcsv, wcsv, args.pmc_command)
        with open(out_md, "w") as f:
            f.write(text)
        print(text)
        return

    if args.summarize_routing_pmc:
        fcsv, wcsv, out_md = args.summarize_routing_pmc
        text = summarize_routing_pmc(fcsv, wcsv, args.pmc_command)
        with open(out_md, "w") as f:
            f.write(text)
        print(text)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the routed stack runs and is timed on a single MI355X; "
              "sharding it over several GPUs is not implemented.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_02829_amd import abi, inputs

    abi.lib()
    torch.cuda.set_device(0)
    w = inputs.WORKLOADS[args.workload]
    if args.generative_only:
        print(json.dumps({"generative": generative_stage(args.steps, max(1, args.steps // 2))}), flush=True)
        return
    if args.copy_probe:
        src = torch.empty(COPY_PROBE_BYTES, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()
    log(f"workload {w.name}: B={w.B} L={w.L} K={w.K} D={w.D} H={w.H} F={w.F} blocks={w.n_blocks} {w.dtype}")

    # ---------------------------------------------------------------- routed (sparse) mode
    torch.cuda.reset_peak_memory_stats()
    base_mem = torch.cuda.memory_allocated()
    sp = Step(w, dense=False, fused=not args.unfused)
    sp.run(0)
    torch.cuda.synchronize()
    sparse_peak = torch.cuda.max_memory_allocated() - base_mem
    breakdown = kernel_breakdown(sp, 1)
    dom = max(breakdown, key=lambda k: breakdown[k]["ms"])
    if args.breakdown:
        tot = sum(v["ms"] for v in breakdown.values())
        for k, v in sorted(breakdown.items(), key=lambda kv: -kv[1]["ms"]):
            log(f"  {k:16s} {v['launches']:5.0f} launches {v['ms']:9.3f} ms ({100 * v['ms'] / tot:5.1f}%)")
    log(f"dominant kernel group: {dom}")
    # timed region: K steps; HIP events bracket only the dominant kernel's launches
    ms_step, ms_gpu, prof = time_steps(sp, args.steps, args.warmup, start=2, profile_filter=dom)
    finite = bool(torch.isfinite(sp.x.float()).all().item() and torch.isfinite(sp.g.float()).all().item())
    graph = None
    if args.graph:
        graph = graph_timing(sp, args.steps, args.warmup)
    del sp
    torch.cuda.empty_cache()

    d = prof[dom]
    per_launch_ms = d["ms"] / d["launches"]
    per_launch_flops = d["flops"] / d["launches"]
    per_launch_bytes = d["bytes"] / d["launches"]
    if per_launch_flops > 0:
        achieved, peak, unit, bound = per_launch_flops / (per_launch_ms * 1e-3), PEAK_BF16_FLOPS, "TFLOP/s", "mfma"
        achieved_u, peak_u = achieved / 1e12, peak / 1e12
    else:
        achieved, peak, unit, bound = per_launch_bytes / (per_launch_ms * 1e-3), PEAK_HBM_BYTES, "GB/s", "hbm"
        achieved_u, peak_u = achieved / 1e9, peak / 1e9
    # the sustained matrix-core rate of this machine (its clock under MFMA load), a second
    # denominator beside the datasheet peak
    sustained = None
    if bound == "mfma":
        sink = torch.empty(4, dtype=torch.float32, device="cuda")
        sustained = abi.sr_probe_mfma_rate(sink)
        torch.cuda.synchronize()

    # whole-stack MFMA fraction: algorithmic block FLOPs per step over step time
    blk_flops = block_flops(w, w.K)

    # ---------------------------------------------------------------- dense keep=100% mode
    dense = None
    if args.dense_steps > 0:
        torch.cuda.reset_peak_memory_stats()
        base_mem = torch.cuda.memory_allocated()
        dn = Step(w, dense=True)
        dn.run(0)
        torch.cuda.synchronize()
        dense_peak = torch.cuda.max_memory_allocated() - base_mem
        dms, _, _ = time_steps(dn, args.dense_steps, 1, start=1)
        dense = {"ms_per_step": round(dms, 3), "peak_bytes": int(dense_peak)}
        del dn
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- whole trunk (2, n-4, 2)
    trunk = None
    if args.trunk_steps > 0 and w.kind == "preln" and w.n_blocks >= 5 and w.backward:
        from paper_2607_02829_amd.trunk import eq_speedup_estimate
        torch.cuda.reset_peak_memory_stats()
        base_mem = torch.cuda.memory_allocated()
        tr = TrunkStep(w)
        tr.run(0)
        torch.cuda.synchronize()
        trunk_peak = torch.cuda.max_memory_allocated() - base_mem
        tms, _, _ = time_steps(tr, args.trunk_steps, 1, start=1)
        n1, n2, n3 = tr.split
        finite_trunk = bool(torch.isfinite(tr.trunk.x3.float()).all().item()
                            and torch.isfinite(tr.trunk.g0.float()).all().item())
        del tr
        torch.cuda.empty_cache()
        # the attention-score selector (top-K by attention received in the last dense-early
        # block) in place of random selection: its overhead per step
        tra = TrunkStep(w, select="attn")
        tra.run(0)
        torch.cuda.synchronize()
        ams, _, _ = time_steps(tra, args.trunk_steps, 1, start=1)
        del tra
        torch.cuda.empty_cache()
        # activation checkpointing: one stage's saved activations at a time, each stage's
        # forward run again before its backward
        torch.cuda.reset_peak_memory_stats()
        base_mem = torch.cuda.memory_allocated()
        trc = TrunkStep(w, checkpoint=True)
        trc.run(0)
        torch.cuda.synchronize()
        ckpt_peak = torch.cuda.max_memory_allocated() - base_mem
        cms, _, _ = time_steps(trc, args.trunk_steps, 1, start=1)
        del trc
        torch.cuda.empty_cache()
        trunk = {"split": list((2, w.n_blocks - 4, 2)), "ms_per_step": round(tms, 3), "peak_bytes": int(trunk_peak),
                 "checkpoint": {"ms_per_step": round(cms, 3), "peak_bytes": int(ckpt_peak),
                                "peak_ratio": round(trunk_peak / ckpt_peak, 3)},
                 "attn_selector_ms_per_step": round(ams, 3), "attn_selector_overhead_ms": round(ams - tms, 3),
                 "speedup_vs_dense": round(dense["ms_per_step"] / tms, 3) if dense else None,
                 "eq_speedup_estimate": round(eq_speedup_estimate((n1, n2, n3), w.keep), 3),
                 "outputs_finite": finite_trunk}
        if not args.no_trunk_sweep:
            trunk["sweep"] = trunk_sweep(w, dense["ms_per_step"] if dense else None)

    # routing kernels: in-step launch times (per-kernel breakdown) and a cache-evicting size sweep
    routing = {"in_step": {}, "sweep": []}
    for name in ("gather", "scatter_delta", "gather_f32", "scatter_f32"):
        if name in breakdown and breakdown[name]["launches"] > 0:
            b = breakdown[name]
            us = b["ms"] / b["launches"] * 1e3
            gbs = b["bytes"] / b["launches"] / (us * 1e-6) / 1e9
            routing["in_step"][name] = {"us": round(us, 2), "GB/s": round(gbs, 1),
                                        "frac_of_8TB/s": round(gbs * 1e9 / PEAK_HBM_BYTES, 3)}
    if w.dtype == "bf16" and not args.no_routing_sweep:
        routing["sweep"] = routing_sweep(w.D)

    workloads = None
    if not args.no_workloads:
        workloads = {n: workload_summary(n) for n in ("b5625", "c1406", "edm") if n != w.name}
    generative = None if args.no_generative else generative_stage()
    xattn = cross_attention_timing() if args.cross_attention else None
    cpu = None if args.no_cpu_baseline else cpu_baseline(w)

    routed_tok_s = w.B * w.K / (ms_step * 1e-3)
    out = {
        "metric": "routed tokens/s fwd+bwd, ms/step at 0.25°-shape; speedup vs dense keep=100%",
        "value": round(routed_tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic (seeded smooth Gaussian random token fields, N(0,0.02) weights)",
        "config": {"workload": f"{w.name}: {w.Hg}x{w.Wg} token grid (L={w.L}), keep 25% (K={w.K}), B={w.B}, "
                               f"D={w.D}, H={w.H}, F={w.F}, {w.n_blocks} {w.kind} blocks, {w.select} selection",
                   "B": w.B, "L": w.L, "K": w.K, "D": w.D, "H": w.H, "F": w.F, "n_blocks": w.n_blocks,
                   "parallelism": "none (1 GPU)"},
        "routed_step_calls": "separate gather / blocks / scatter" if args.unfused else "fused (sr_routed_blocks_fwd/bwd)",
        "gpu_ms_per_step_events": round(ms_gpu, 4),
        "full_grid_tokens_per_s": round(w.B * w.L / (ms_step * 1e-3), 1),
        "stack_mfma_frac": round(blk_flops / (ms_step * 1e-3) / PEAK_BF16_FLOPS, 4),
        "dense": dense,
        "speedup_vs_dense": round(dense["ms_per_step"] / ms_step, 3) if dense else None,
        "trunk": trunk,
        "workloads": workloads,
        "generative": generative,
        "graph": graph,
        "cross_attention": xattn,
        "peak_bytes": {"sparse": int(sparse_peak), "dense": dense["peak_bytes"] if dense else None,
                       "ratio": round(dense["peak_bytes"] / sparse_peak, 3) if dense else None},
        "roofline": {"kernel": dom, "bound": bound, "achieved": round(achieved_u, 2), "peak": peak_u, "unit": unit,
                     "frac": round(achieved / peak, 4), "traffic": traffic_for(dom, w.name),
                     "launches_timed": int(d["launches"]), "avg_launch_us": round(per_launch_ms * 1e3, 2),
                     "peak_sustained": round(sustained, 1) if sustained else None,
                     "frac_sustained": round(achieved_u / sustained, 4) if sustained else None},
        "cpu_baseline": cpu,
        "routing_bandwidth": routing,
        "outputs_finite": finite,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
