"""The whole block trunk with a dense-sparse-dense split (Sec. 3.2 "Three-stage block
partition", Eq. partition; Alg. 1).

A trunk of n1 + n2 + n3 pre-LN blocks runs its n1 early blocks densely on all L
tokens, its n2 middle blocks on K routed tokens per sample (random selection, or
top-K by attention received in the last early block; gather, blocks,
residual-delta scatter into the early blocks' output), and its
n3 late blocks densely again; the backward runs the three stages in reverse,
with the routing VJP (gather of the gradient, the middle blocks' VJP, scatter of
the gradient delta) between the two dense ones.  The split of the deterministic
forecaster is (2, 8, 2) (Sec. 4.1, deterministic model; App. A.1); Eq. speedup
(Sec. 3.2) estimates the trunk speedup over the dense trunk as N / (n1 + n2 r^2 + n3),
counting attention cost only.

Orchestration only: every step is a libsr entry point enqueued on the caller's
current stream; the three stages have their own configs, parameters, gradients
and saved activations and share one scratch buffer (their calls are ordered on
the stream, and each backward joins its second stream before it returns).

Activation checkpointing (optional; the paper trains with it to bound peak memory,
Sec. 4.1 and App. A.2 "Training Configuration"): the three stages then share one
saved-activation buffer, sized for the largest, and the backward re-runs each stage's
forward from that stage's input (x0, the gathered tokens h0, the scattered x1, all kept)
right before the stage's backward.  The kernels are deterministic, so the recomputed
activations, and with them every gradient, are bit for bit those of the run without
checkpointing; the price is one more forward of every block.
"""
from __future__ import annotations

from . import abi, device


def eq_speedup_estimate(split, keep: float) -> float:
    """Attention-cost estimate of the trunk's speedup over the same blocks on all tokens
    (Sec. 3.2, Eq. (speedup)): N / (n1 + n2 r^2 + n3) with N = n1 + n2 + n3; only the middle
    blocks' attention is counted as shrinking, by r^2."""
    n1, n2, n3 = (int(v) for v in split)
    if min(n1, n2, n3) < 0 or n1 + n2 + n3 < 1:
        raise ValueError(f"split {split} needs non-negative block counts and at least one block")
    if not 0.0 < keep <= 1.0:
        raise ValueError(f"keep ratio {keep} not in (0, 1]")
    return (n1 + n2 + n3) / (n1 + n2 * keep * keep + n3)


class Trunk:
    """Device buffers and the launch sequence of one trunk forward + backward.

    ``params_storage``: n1 + n2 + n3 per-block storage dicts (early, middle, late).
    The dense stages read and write whole (B, L, D) sequences; the routed stage
    scatters into the early stage's output in place, which is then the late
    stage's input."""

    def __init__(self, w, split, params_storage, K: int | None = None, seed: int = 42, select: str = "random",
                 checkpoint: bool = False):
        """``select``: "random" (the method's selector) or "attn" (top-K by the attention each
        token receives in the last dense-early block, summed over heads: the paper's
        attention-score ablation).  ``checkpoint``: keep one stage's saved activations at a
        time and recompute them in the backward."""
        import torch
        n1, n2, n3 = split
        if min(n1, n2, n3) < 1:
            raise ValueError(f"split {split}: every stage needs at least one block")
        if len(params_storage) != n1 + n2 + n3:
            raise ValueError(f"{len(params_storage)} blocks of parameters for split {split}")
        if w.kind != "preln":
            raise ValueError("the trunk is built for pre-LN blocks")
        if select not in ("random", "attn"):
            raise ValueError(f"unknown selector {select!r}")
        if not isinstance(checkpoint, bool):
            raise ValueError(f"checkpoint must be True or False, not {checkpoint!r}")
        self.w, self.split, self.seed, self.select = w, tuple(split), seed, select
        self.checkpoint = checkpoint
        self.K = w.K if K is None else K
        if not 1 <= self.K <= w.L:
            raise ValueError(f"K={self.K} outside [1, L={w.L}]")
        self.cfg = [device.config_for(w, n_blocks=n) for n in split]
        bounds = (0, n1, n1 + n2, n1 + n2 + n3)
        self.params = [device.DeviceParams(params_storage[bounds[i]:bounds[i + 1]], w.kind) for i in range(3)]
        self.grads = [device.DeviceGrads(w, n, skip_unused=True) for n in split]
        S = (w.L, self.K, w.L)
        sizes = [abi.sr_workspace_bytes(c, s) for c, s in zip(self.cfg, S)]
        scratch_bytes = max([16] + [cb for _, cb in sizes])
        if checkpoint:
            shared = torch.empty(max([16] + [sb for sb, _ in sizes]), dtype=torch.uint8, device="cuda")
            self.saved = [shared, shared, shared]
        else:
            self.saved = [torch.empty(max(sb, 16), dtype=torch.uint8, device="cuda") for sb, _ in sizes]
        self.scratch = torch.empty(scratch_bytes, dtype=torch.uint8, device="cuda")
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        B, L, D, K = w.B, w.L, w.D, self.K
        self.x1 = torch.empty((B, L, D), dtype=dt, device="cuda")     # early output; routed stage writes into it
        self.x3 = torch.empty_like(self.x1)                            # trunk output
        self.g2 = torch.empty_like(self.x1)                            # late-stage input gradient, then dx of x1
        self.g0 = torch.empty_like(self.x1)                            # trunk input gradient
        self.idx = torch.empty((B, K), dtype=torch.int32, device="cuda")
        self.h0 = torch.empty((B, K, D), dtype=dt, device="cuda")
        self.h = torch.empty_like(self.h0)
        self.gh = torch.empty_like(self.h0)
        self.dh = torch.empty_like(self.h0)
        self.colsum = (torch.empty((B, w.H, L), dtype=torch.float32, device="cuda") if select == "attn" else None)

    def forward(self, x0, step: int):
        """x0: (B, L, D) storage tensor (not modified; with checkpointing the backward reads it
        again, so it must keep its values until then).  Returns the trunk output x3."""
        a, (ce, cm, cl), (pe, pm, pl) = abi, self.cfg, self.params
        K = self.K
        self.x0 = x0
        a.sr_dense_blocks_fwd(ce, pe.array, None, x0, self.x1, self.saved[0], self.scratch)
        if self.select == "attn":
            a.sr_attention_colsums(ce, self.w.L, self.saved[0], self.split[0] - 1, self.colsum)
            a.sr_select_topk_scores(cm, K, self.colsum, self.w.H, self.idx)
        else:
            a.sr_select_indices(cm, K, a.SR_SEL_RANDOM, self.seed, step, None, None, self.idx)
        a.sr_gather(cm, K, self.x1, self.idx, self.h0)
        a.sr_sparse_blocks_fwd(cm, K, pm.array, None, self.h0, self.h, self.saved[1], self.scratch)
        a.sr_scatter_delta(cm, K, self.x1, self.h, self.h0, self.idx)
        a.sr_dense_blocks_fwd(cl, pl.array, None, self.x1, self.x3, self.saved[2], self.scratch)
        return self.x3

    def backward(self, g3):
        """g3: (B, L, D) storage gradient of the trunk output (not modified).  Returns the
        input gradient g0; the parameter gradients are in ``self.grads`` (early, middle, late)."""
        a, (ce, cm, cl), (pe, pm, pl) = abi, self.cfg, self.params
        ge, gm, gl = (g.array for g in self.grads)
        K, ck = self.K, self.checkpoint
        # with checkpointing each stage's forward runs again first, from the stage's kept input;
        # its output goes to g0 (or to h, which holds the same bits), which the early stage's
        # backward overwrites last
        if ck:
            a.sr_dense_blocks_fwd(cl, pl.array, None, self.x1, self.g0, self.saved[2], self.scratch)
        a.sr_dense_blocks_bwd(cl, pl.array, None, self.saved[2], g3, self.g2, gl, None, self.scratch)
        a.sr_gather(cm, K, self.g2, self.idx, self.gh)
        if ck:
            a.sr_sparse_blocks_fwd(cm, K, pm.array, None, self.h0, self.h, self.saved[1], self.scratch)
        a.sr_sparse_blocks_bwd(cm, K, pm.array, None, self.saved[1], self.gh, self.dh, gm, None, self.scratch)
        a.sr_scatter_delta(cm, K, self.g2, self.dh, None, self.idx)
        if ck:
            a.sr_dense_blocks_fwd(ce, pe.array, None, self.x0, self.g0, self.saved[0], self.scratch)
        a.sr_dense_blocks_bwd(ce, pe.array, None, self.saved[0], self.g2, self.g0, ge, None, self.scratch)
        return self.g0

    def block_grads(self):
        """The fp32 gradient tensors of all n1 + n2 + n3 blocks, in trunk order."""
        return [g for stage in self.grads for g in stage.tensors]
