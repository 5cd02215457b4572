"""Gather and residual-delta scatter (Sec. 3.2 "Residual delta formulation",
Eq. scatter; Alg. 1 gather/scatter steps; App. A.4).

gather:   h0[b, k, :] = x[b, I[b, k], :]                      (a copy of bits)
scatter:  x'[b, i, :] = x0[b, i, :] + Delta[b, k, :]  for i = I[b, k],
          Delta = h - h0, and x'[b, i, :] = x0[b, i, :] exactly for every
          unselected i (the paper's "retain x0 exactly").

Precision reading (the paper materialises Delta in the model dtype and adds it
in place, which under bf16 rounds twice): Delta is formed in fp32 and the sum is
rounded once to the storage type,

    x'[b,i,d] = rnd( f32(x0[b,i,d]) + ( f32(h[b,k,d]) - f32(h0[b,k,d]) ) ),

fp32 subtract first, then fp32 add (no fused multiply-add), each IEEE
round-to-nearest-even, then one RNE rounding to bf16 for bf16 storage.
With ``h0`` omitted the gathered rows are re-read from x0 itself, which is the
same value by the definition of gather.

Index sets are per sample (B, K) (the text's "per sample"); ``shared=True`` uses
row 0 for every sample (the App. A.4 listing's single index vector).

Pins: unselected rows bit-identical to x0; h == h0 leaves x bit-identical; a
one-element hand-computed rounding case; gather against plain integer indexing
semantics on a permutation (gather then scatter of an identity stack).
"""
from __future__ import annotations

import numpy as np

from .numerics import storage_to_f32, f32_to_storage


def _row(idx: np.ndarray, b: int, shared: bool) -> np.ndarray:
    return idx[0] if shared else idx[b]


def gather(x: np.ndarray, idx: np.ndarray, shared: bool = False) -> np.ndarray:
    x = np.asarray(x)
    B = x.shape[0]
    K = idx.shape[1]
    out = np.empty((B, K) + x.shape[2:], dtype=x.dtype)
    for b in range(B):
        for k, i in enumerate(_row(idx, b, shared)):
            out[b, k] = x[b, int(i)]
    return out


def scatter_delta(x0: np.ndarray, h: np.ndarray, h0: np.ndarray | None, idx: np.ndarray,
                  shared: bool = False) -> np.ndarray:
    """Returns x' (a new array); x0 is not modified."""
    x0 = np.asarray(x0)
    out = x0.copy()
    B = x0.shape[0]
    for b in range(B):
        for k, i in enumerate(_row(idx, b, shared)):
            i = int(i)
            base = storage_to_f32(x0[b, i])
            hv = storage_to_f32(h[b, k])
            h0v = storage_to_f32(x0[b, i] if h0 is None else h0[b, k])
            delta = (hv - h0v).astype(np.float32)
            out[b, i] = f32_to_storage((base + delta).astype(np.float32), x0)
    return out
