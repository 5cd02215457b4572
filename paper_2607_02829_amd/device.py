"""Device-memory helpers for callers of the binding: upload seeded host arrays to
GPU tensors and fill the ABI's parameter / gradient structs.  Marshalling only:
every step of the hot path runs in libsr's kernels."""
from __future__ import annotations

import ctypes

import numpy as np

from . import abi


def config_for(w, dtype: str | None = None, n_blocks: int | None = None, idx_shared: int = 0,
               eps: float = 1e-6) -> abi.SrConfig:
    dt = w.dtype if dtype is None else dtype
    return abi.SrConfig(B=w.B, L=w.L, D=w.D, H=w.H, F=w.F,
                        n_blocks=w.n_blocks if n_blocks is None else n_blocks,
                        dtype=abi.SR_BF16 if dt == "bf16" else abi.SR_F32,
                        kind=abi.SR_BLOCK_ADALN if w.kind == "adaln" else abi.SR_BLOCK_PRELN,
                        ln_eps=eps, idx_shared=idx_shared)


def to_device(a: np.ndarray, device="cuda"):
    """Host storage array (float32, or uint16 bf16 bits, or int32) -> GPU tensor."""
    import torch
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(a)
    return t.to(device)


def to_host(t) -> np.ndarray:
    """GPU tensor -> host array in the same representation as ``to_device``'s input."""
    import torch
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


class DeviceParams:
    """Block parameters on the GPU plus the host array of sr_block_params."""

    def __init__(self, params_storage: list[dict[str, np.ndarray]], kind: str, device="cuda"):
        self.tensors = [{k: to_device(v, device) for k, v in p.items()} for p in params_storage]
        n = len(self.tensors)
        self.array = (abi.SrBlockParams * n)()
        for i, p in enumerate(self.tensors):
            for name in abi.PARAM_FIELDS:
                unused = (kind == "preln" and name in ("w_ada", "b_ada")) or (kind == "adaln" and name.startswith("ln"))
                use = not unused
                setattr(self.array[i], name, p[name].data_ptr() if use else None)


class DeviceGrads:
    """fp32 gradient buffers for n blocks plus the host array of sr_block_grads."""

    def __init__(self, w, n_blocks: int, device="cuda", skip_unused: bool = False):
        """``skip_unused`` passes NULL for the gradients of parameters the block kind does not
        read (otherwise the library fills them with zeros)."""
        import torch
        D, F = w.D, w.F
        shapes = {"ln1_w": (D,), "ln1_b": (D,), "w_qkv": (3 * D, D), "b_qkv": (3 * D,), "w_o": (D, D),
                  "b_o": (D,), "ln2_w": (D,), "ln2_b": (D,), "w_fc1": (F, D), "b_fc1": (F,),
                  "w_fc2": (D, F), "b_fc2": (D,), "w_ada": (6 * D, D), "b_ada": (6 * D,)}
        self.tensors = [{k: torch.full(s, float("nan"), dtype=torch.float32, device=device)
                         for k, s in shapes.items()} for _ in range(n_blocks)]
        self.array = (abi.SrBlockGrads * n_blocks)()
        for i, g in enumerate(self.tensors):
            for name in abi.PARAM_FIELDS:
                unused = (w.kind == "preln" and name in ("w_ada", "b_ada")) or (w.kind == "adaln" and name.startswith("ln"))
                setattr(self.array[i], name, None if (skip_unused and unused) else g[name].data_ptr())


def workspace(cfg: abi.SrConfig, S: int, device="cuda"):
    """(saved, scratch) uint8 GPU tensors sized by sr_workspace_bytes."""
    import torch
    sb, cb = abi.sr_workspace_bytes(cfg, S)
    return (torch.empty(max(sb, 16), dtype=torch.uint8, device=device),
            torch.empty(max(cb, 16), dtype=torch.uint8, device=device))


class DeviceEdmParams:
    """Generative-block parameters on the GPU plus the host array of sr_edm_block_params."""

    def __init__(self, params_storage: list[dict[str, np.ndarray]], device="cuda"):
        self.tensors = [{k: to_device(v, device) for k, v in p.items()} for p in params_storage]
        self.array = (abi.SrEdmBlockParams * len(self.tensors))()
        for i, p in enumerate(self.tensors):
            for name in abi.EDM_PARAM_FIELDS:
                setattr(self.array[i], name, p[name].data_ptr())


class DeviceEdmGrads:
    """fp32 gradient buffers of n generative blocks plus the host array of sr_edm_block_grads."""

    def __init__(self, D: int, F: int, n_blocks: int, device="cuda"):
        import torch
        shapes = edm_param_shapes(D, F)
        self.tensors = [{k: torch.full(s, float("nan"), dtype=torch.float32, device=device)
                         for k, s in shapes.items()} for _ in range(n_blocks)]
        self.array = (abi.SrEdmBlockGrads * n_blocks)()
        for i, g in enumerate(self.tensors):
            for name in abi.EDM_PARAM_FIELDS:
                setattr(self.array[i], name, g[name].data_ptr())


def edm_param_shapes(D: int, F: int) -> dict[str, tuple[int, ...]]:
    return {"w_film": (2 * D, D), "b_film": (2 * D,), "w_qkv": (3 * D, D), "b_qkv": (3 * D,), "w_o": (D, D),
            "b_o": (D,), "lnc_w": (D,), "lnc_b": (D,), "w_q": (D, D), "b_q": (D,), "w_kv": (2 * D, D),
            "b_kv": (2 * D,), "w_oc": (D, D), "b_oc": (D,), "w_g": (D, D), "b_g": (D,), "ln2_w": (D,),
            "ln2_b": (D,), "w_fc1": (F, D), "b_fc1": (F,), "w_fc2": (D, F), "b_fc2": (D,)}


def edm_workspace(cfg: abi.SrConfig, S: int, device="cuda"):
    """(saved, scratch) uint8 GPU tensors sized by sr_edm_workspace_bytes."""
    import torch
    sb, cb = abi.sr_edm_workspace_bytes(cfg, S)
    return (torch.empty(max(sb, 16), dtype=torch.uint8, device=device),
            torch.empty(max(cb, 16), dtype=torch.uint8, device=device))
