"""Seeded synthetic inputs for the routed middle-block stack.

This module only draws random numbers and shapes them; it computes nothing of
the method itself.  Both the HIP path and the CPU oracle receive exactly the
arrays produced here.

Workloads (token grids follow Sec. 4.1 "Dataset" and the architecture tables in
App. A.1; the middle-stack sizes are the ones the benchmark measures):

=====  ======  =========================  =====  ====  ==  ===  ====  ==  ======  ==========
name   B       grid (tokens)              L      K     D   H    F     n2  dtype   selection
=====  ======  =========================  =====  ====  ==  ===  ====  ==  ======  ==========
tiny   1       8 x 16                     128    32    128 4    512   2   f32     random
b5625  8       16 x 32  (5.625 deg, p=2)  512    128   1024 16  4096  8   bf16    random
c1406  2       64 x 128 (1.40625 deg, p=2) 8192  2048  1024 16  4096  8   bf16    random
d025   1       90 x 180 (0.25 deg, p=8)   16200  4050  1024 16  4096  12  bf16    random
edm    2       64 x 128                   8192   2048  1024 16  4096  8   bf16    top-k (adaLN)
gen    2       64 x 128                   8192   2048  1024 8   4096  4   bf16    random (generative
                                                                                block, Z_c of L tokens)
=====  ======  =========================  =====  ====  ==  ===  ====  ==  ======  ==========

Token fields stand in for ERA5 (not available): a smooth Gaussian random field
on the token grid (white noise filtered by a separable Gaussian, periodic in
longitude, reflecting at the poles, standardised per channel), or for ``tiny``
N(0,1) noise plus low-frequency sinusoids.  Weights are N(0, 0.02), biases 0,
LayerNorm gamma=1 / beta=0 unless ``randomise_affine`` asks for random values
(used by gradient tests so every parameter path carries signal).
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

BLOCK_PARAM_NAMES = (
    "ln1_w", "ln1_b", "w_qkv", "b_qkv", "w_o", "b_o",
    "ln2_w", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2", "w_ada", "b_ada",
)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hg: int          # token-grid rows (latitude)
    Wg: int          # token-grid columns (longitude)
    D: int
    H: int
    F: int
    n_blocks: int
    keep: float
    dtype: str       # "f32" | "bf16"  (storage type; accumulation is always fp32)
    kind: str        # "preln" | "adaln" | "edm" (the generative model's block)
    select: str      # "random" | "topk"
    ell: float       # correlation length of the token field, in tokens
    backward: bool
    seed: int

    @property
    def L(self) -> int:
        return self.Hg * self.Wg

    @property
    def K(self) -> int:
        # K = floor(L * r) (Sec. 3.2, "Random token selection"), computed in double.
        return int(math.floor(self.L * self.keep))

    @property
    def hd(self) -> int:
        return self.D // self.H

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", 1, 8, 16, 128, 4, 512, 2, 0.25, "f32", "preln", "random", 0.0, False, 0),
    "b5625": Workload("b5625", 8, 16, 32, 1024, 16, 4096, 8, 0.25, "bf16", "preln", "random", 4.0, True, 1),
    "c1406": Workload("c1406", 2, 64, 128, 1024, 16, 4096, 8, 0.25, "bf16", "preln", "random", 4.0, True, 2),
    "d025": Workload("d025", 1, 90, 180, 1024, 16, 4096, 12, 0.25, "bf16", "preln", "random", 6.0, True, 3),
    "edm": Workload("edm", 2, 64, 128, 1024, 16, 4096, 8, 0.25, "bf16", "adaln", "topk", 4.0, True, 4),
    # the generative model's sparse middle stage (App. A.1 EDM table: D = 1024, 8 heads of 128,
    # split (2, 4, 2)) on the 1.40625 deg token grid: 4 blocks on K = 2048 routed tokens with
    # cross-attention to all 8192 conditioning tokens
    "gen": Workload("gen", 2, 64, 128, 1024, 8, 4096, 4, 0.25, "bf16", "edm", "random", 4.0, True, 5),
}


def small(name: str = "small", **kw) -> Workload:
    """A small workload for quick parity runs (several tiles and a ragged tail)."""
    base = Workload(name, 2, 10, 20, 256, 4, 1024, 2, 0.25, "bf16", "preln", "random", 3.0, True, 7)
    return base.with_(**kw)


# ----------------------------------------------------------------------------------
# storage conversion (input preparation only)
# ----------------------------------------------------------------------------------

def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    """fp32 array -> storage array: float32 for "f32"; uint16 bf16 bits (RNE) for "bf16"."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "f32":
        return a
    import torch
    t = torch.from_numpy(a).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def storage_nbytes(dtype: str) -> int:
    return 4 if dtype == "f32" else 2


# ----------------------------------------------------------------------------------
# token fields
# ----------------------------------------------------------------------------------

def _grf(rng: np.random.Generator, B: int, Hg: int, Wg: int, D: int, ell: float) -> np.ndarray:
    from scipy.ndimage import gaussian_filter1d
    z = rng.standard_normal((B, Hg, Wg, D), dtype=np.float32)
    sig = ell / 2.0
    if sig > 0:
        z = gaussian_filter1d(z, sig, axis=1, mode="reflect")   # poles: reflect
        z = gaussian_filter1d(z, sig, axis=2, mode="wrap")      # longitude: periodic
    mu = z.mean(axis=(0, 1, 2), keepdims=True)
    sd = z.std(axis=(0, 1, 2), keepdims=True)
    z = (z - mu) / np.maximum(sd, 1e-6)
    return z.reshape(B, Hg * Wg, D).astype(np.float32)


def _sinusoid_field(rng: np.random.Generator, B: int, Hg: int, Wg: int, D: int) -> np.ndarray:
    r = np.arange(Hg, dtype=np.float64)[:, None]
    c = np.arange(Wg, dtype=np.float64)[None, :]
    out = rng.standard_normal((B, Hg, Wg, D)).astype(np.float64)
    fr = rng.integers(1, 3, size=D)
    fc = rng.integers(1, 3, size=D)
    ph = rng.uniform(0, 2 * np.pi, size=D)
    for d in range(D):
        out[:, :, :, d] += np.sin(2 * np.pi * (fr[d] * r / Hg + fc[d] * c / Wg) + ph[d])
    return out.reshape(B, Hg * Wg, D).astype(np.float32)


def token_field(w: Workload, which: int = 0) -> np.ndarray:
    """(B, L, D) fp32 token sequence; ``which`` selects an independent field."""
    rng = np.random.default_rng([1000 + w.seed, which])
    if w.ell <= 0:
        return _sinusoid_field(rng, w.B, w.Hg, w.Wg, w.D)
    return _grf(rng, w.B, w.Hg, w.Wg, w.D, w.ell)


def upstream_grad(w: Workload, rows: int | None = None) -> np.ndarray:
    """N(0,1) gradient dL/dx' of shape (B, L, D) (or (B, rows, D))."""
    rng = np.random.default_rng([3000 + w.seed])
    n = w.L if rows is None else rows
    return rng.standard_normal((w.B, n, w.D), dtype=np.float32)


def cond_vector(w: Workload) -> np.ndarray:
    """Per-sample conditioning vector c ~ N(0,1), shape (B, D) (adaLN blocks)."""
    rng = np.random.default_rng([4000 + w.seed])
    return rng.standard_normal((w.B, w.D), dtype=np.float32)


def block_params(w: Workload, n_blocks: int | None = None, randomise_affine: bool = False,
                 zero: tuple[str, ...] = (), std: float = 0.02) -> list[dict[str, np.ndarray]]:
    """Per-block parameters in nn.Linear layout ([out, in]), fp32.

    ``zero`` lists parameter names to set to zero (invariant tests)."""
    D, F = w.D, w.F
    nb = w.n_blocks if n_blocks is None else n_blocks
    shapes = {
        "ln1_w": (D,), "ln1_b": (D,), "w_qkv": (3 * D, D), "b_qkv": (3 * D,),
        "w_o": (D, D), "b_o": (D,), "ln2_w": (D,), "ln2_b": (D,),
        "w_fc1": (F, D), "b_fc1": (F,), "w_fc2": (D, F), "b_fc2": (D,),
        "w_ada": (6 * D, D), "b_ada": (6 * D,),
    }
    out = []
    for i in range(nb):
        rng = np.random.default_rng([2000 + w.seed, i])
        p = {}
        for name in BLOCK_PARAM_NAMES:
            shp = shapes[name]
            if name.startswith("w_"):
                v = rng.normal(0.0, std, size=shp)
            elif name in ("ln1_w", "ln2_w"):
                v = 1.0 + (rng.normal(0.0, 0.1, size=shp) if randomise_affine else 0.0) * np.ones(shp)
            else:
                v = rng.normal(0.0, 0.05, size=shp) if randomise_affine else np.zeros(shp)
            if name in zero:
                v = np.zeros(shp)
            p[name] = np.asarray(v, dtype=np.float32)
        out.append(p)
    return out


EDM_PARAM_NAMES = (
    "w_film", "b_film", "w_qkv", "b_qkv", "w_o", "b_o",
    "lnc_w", "lnc_b", "w_q", "b_q", "w_kv", "b_kv", "w_oc", "b_oc", "w_g", "b_g",
    "ln2_w", "ln2_b", "w_fc1", "b_fc1", "w_fc2", "b_fc2",
)


def edm_block_params(w: Workload, n_blocks: int | None = None, randomise_affine: bool = False,
                     std: float = 0.02) -> list[dict[str, np.ndarray]]:
    """Parameters of the generative model's blocks ([out, in] layout, fp32): linear weights
    N(0, std), biases 0, LayerNorm gamma = 1 and beta = 0 unless ``randomise_affine`` (then
    biases and beta N(0, 0.05), gamma 1 + N(0, 0.1), so every gradient path carries signal)."""
    D, F = w.D, w.F
    nb = w.n_blocks if n_blocks is None else n_blocks
    shapes = {"w_film": (2 * D, D), "b_film": (2 * D,), "w_qkv": (3 * D, D), "b_qkv": (3 * D,),
              "w_o": (D, D), "b_o": (D,), "lnc_w": (D,), "lnc_b": (D,), "w_q": (D, D), "b_q": (D,),
              "w_kv": (2 * D, D), "b_kv": (2 * D,), "w_oc": (D, D), "b_oc": (D,), "w_g": (D, D), "b_g": (D,),
              "ln2_w": (D,), "ln2_b": (D,), "w_fc1": (F, D), "b_fc1": (F,), "w_fc2": (D, F), "b_fc2": (D,)}
    out = []
    for i in range(nb):
        rng = np.random.default_rng([5000 + w.seed, i])
        p = {}
        for name in EDM_PARAM_NAMES:
            shp = shapes[name]
            if name.startswith("w_"):
                v = rng.normal(0.0, std, size=shp)
            elif name in ("lnc_w", "ln2_w"):
                v = 1.0 + (rng.normal(0.0, 0.1, size=shp) if randomise_affine else np.zeros(shp))
            else:
                v = rng.normal(0.0, 0.05, size=shp) if randomise_affine else np.zeros(shp)
            p[name] = np.asarray(v, dtype=np.float32)
        out.append(p)
    return out


def noise_embedding(w: Workload) -> np.ndarray:
    """Stand-in for the noise embedding e_sigma, one global vector per sample: N(0,1) of shape
    (B, D) (the embedding MLP of ln(sigma) is not on the path)."""
    rng = np.random.default_rng([6000 + w.seed])
    return rng.standard_normal((w.B, w.D), dtype=np.float32)


def conditioning_tokens(w: Workload) -> np.ndarray:
    """Conditioning sequence Z_c (B, L, D): an independent smooth field on the same token grid
    (the history frames' tokens)."""
    return token_field(w, 2)


def params_to_storage(params: list[dict[str, np.ndarray]], dtype: str) -> list[dict[str, np.ndarray]]:
    return [{k: to_storage(v, dtype) for k, v in p.items()} for p in params]
