"""Token selection (Sec. 3.2 "Random token selection"; Alg. 1, selection step;
App. A.4 code listing), and the deterministic top-k variant.

Random selection
----------------
The paper draws I = sort(randperm(L)[:K]) per sample: K = floor(L*r) indices,
uniform without replacement, returned in ascending order, with a fresh draw at
every forward pass (Sec. 3.4 "Training and inference").  ``randperm`` is not
defined outside PyTorch, so the draw is fixed here by a counter-based generator:
SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014).  Its n-th output from state s is
mix(s + n*gamma) with gamma = 0x9E3779B97F4A7C15 and mix the published 64-bit
finaliser.  For sample b, draw ``step`` and token i:

    s_step = mix(seed   + (step + 1) * gamma)
    s_b    = mix(s_step + (b    + 1) * gamma)
    key_i  = mix(s_b    + (i    + 1) * gamma)          (all mod 2^64)

Sorting the L tokens by key gives a uniformly random permutation (the keys are
distinct because mix is a bijection), so taking its first K entries and sorting
them is randperm(L)[:K].sort().  Equivalently: I = the K tokens with the
smallest keys, ascending.

Pins: mix against SplitMix64's published output stream for seed 1234567;
selection invariants (K entries, strictly increasing, in range, K = L gives all
tokens); uniformity of inclusion (chi-square over many draws); pairwise
inclusion frequency K(K-1)/(L(L-1)) (no-replacement law).

Top-k selection (deterministic routing ablation, App. "regularization
decomposition"; the workload's selector)
------------------------------------------------------------------------------
score_i = sum_d (x_t[i,d] - x_prev[i,d])^2, the squared L2 norm of the
frame difference (ranking by the square equals ranking by the norm).  The
K tokens with the largest scores are kept, ties go to the lower token index,
output ascending.  The score decides an integer result, so its fp32 evaluation
order is part of the definition (both sides evaluate it identically):

  * d_e = fl32(fl32(x_t) - fl32(x_prev)),  q_e = fl32(d_e * d_e)  (no fused multiply-add);
  * elements are taken in 16-byte chunks of 8 bf16 (4 fp32): chunk c = floor(d / V),
    V = 8 (bf16) or 4 (fp32);  chunk c belongs to lane c mod 64, round floor(c / 64);
  * each of the 64 lanes sums its q_e sequentially, rounds ascending, elements of a
    chunk ascending, acc = fl32(acc + q_e), starting from +0;
  * the 64 lane sums are combined by a butterfly: for o = 32,16,8,4,2,1,
    a[l] = fl32(a[l] + a[l xor o]); the result is a[0] (all lanes agree).

Pins: the result lies within the fp32 summation error bound of the exact fp64
sum; fp64-ranked brute force gives the same set when no near-tie exists; planted
exact ties resolve to the lower index; K = L keeps all tokens; a hand-computed
case where the butterfly order changes the fp32 result.

Attention-score selection (Sec. 4.4 "Random vs. learned token selection";
Tab. selection: keep the tokens the final dense-early block attends to most)
----------------------------------------------------------------------------
The paper names the selector but not the score.  Reading taken: the score of
token j is the attention it receives, a_j = sum_h sum_i P_h[i, j], with P_h the
softmax(q k^T / sqrt(hd)) of head h of that block's forward over all S tokens.
``attention_colsums`` gives the per-head column sums colsum[b, h, j] in fp64.
The ranking takes per-head planes in fp32 and adds them in head order from +0
(the planes the HIP path computes are the input of its selection, so the order
of that fp32 sum is part of the definition); then the K largest, ties to the
lower index, ascending, as for the top-k selector above.

Pins: every row of P sums to 1, so each head's column sums add up to S; zero
queries give uniform rows, so every column sum is 1; a loop-written softmax on a
tiny case; permuting the tokens permutes the column sums; planted ties in the
planes resolve to the lower index; one plane reduces to the top-k ranking.
"""
from __future__ import annotations

import numpy as np

from .numerics import storage_to_f32

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def mix64(z):
    """SplitMix64 output finaliser (a bijection on 64-bit words)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def splitmix64_stream(seed: int, n: int) -> np.ndarray:
    """First n outputs of SplitMix64 started from state ``seed``."""
    with np.errstate(over="ignore"):
        st = np.uint64(seed) + np.arange(1, n + 1, dtype=np.uint64) * GAMMA
    return mix64(st)


def random_keys(L: int, b: int, seed: int, step: int) -> np.ndarray:
    with np.errstate(over="ignore"):
        s_step = mix64(np.uint64(seed) + np.uint64(step + 1) * GAMMA)
        s_b = mix64(s_step + np.uint64(b + 1) * GAMMA)
        i = np.arange(L, dtype=np.uint64)
        return mix64(s_b + (i + np.uint64(1)) * GAMMA)


def select_random(B: int, L: int, K: int, seed: int, step: int) -> np.ndarray:
    """(B, K) int32: per sample, sort(randperm(L)[:K]) with the keyed permutation above."""
    if not 0 <= K <= L:
        raise ValueError("need 0 <= K <= L")
    out = np.empty((B, K), dtype=np.int32)
    for b in range(B):
        keys = random_keys(L, b, seed, step)
        perm = np.argsort(keys, kind="stable")      # a uniformly random permutation of 0..L-1
        out[b] = np.sort(perm[:K])
    return out


def topk_score(x_t: np.ndarray, x_prev: np.ndarray) -> np.ndarray:
    """(B, L) fp32 score in the evaluation order stated in the module header."""
    a = storage_to_f32(x_t)
    p = storage_to_f32(x_prev)
    B, L, D = a.shape
    V = 8 if np.asarray(x_t).dtype == np.uint16 else 4
    if D % V:
        raise ValueError("D must be a multiple of the 16-byte chunk")
    d = (a - p).astype(np.float32)
    q = (d * d).astype(np.float32)                  # separate multiply and add, each rounded to fp32
    nchunk = D // V
    lanes = np.zeros((B, L, 64), dtype=np.float32)
    for c in range(nchunk):                           # chunk c: lane c % 64, round c // 64 (rounds ascend)
        lane = c % 64
        for e in range(V):
            lanes[:, :, lane] = lanes[:, :, lane] + q[:, :, c * V + e]
    lane_idx = np.arange(64)
    for o in (32, 16, 8, 4, 2, 1):
        lanes = (lanes + lanes[:, :, lane_idx ^ o]).astype(np.float32)
    return lanes[:, :, 0].copy()


def select_topk(x_t: np.ndarray, x_prev: np.ndarray, K: int) -> np.ndarray:
    """(B, K) int32: the K largest scores, ties to the lower index, ascending."""
    return _largest_k(topk_score(x_t, x_prev), K)


def attention_colsums(q: np.ndarray, k: np.ndarray) -> np.ndarray:
    """q, k: (B, H, S, hd) fp64, a block's queries and keys.  Returns (B, H, S) fp64:
    colsum[b, h, j] = sum_i softmax_j(q_i . k_j / sqrt(hd))."""
    B, H, S, hd = q.shape
    out = np.empty((B, H, S), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            s = q[b, h] @ k[b, h].T / np.sqrt(hd)
            e = np.exp(s - s.max(axis=1, keepdims=True))
            P = e / e.sum(axis=1, keepdims=True)
            out[b, h] = P.sum(axis=0)
    return out


def planes_score(planes: np.ndarray) -> np.ndarray:
    """planes: (B, parts, L) float32 -> (B, L) float32, summed in plane order from +0."""
    planes = np.asarray(planes, dtype=np.float32)
    s = np.zeros((planes.shape[0], planes.shape[2]), dtype=np.float32)
    for p in range(planes.shape[1]):
        s = (s + planes[:, p]).astype(np.float32)
    return s


def select_topk_planes(planes: np.ndarray, K: int) -> np.ndarray:
    """(B, K) int32: the K largest plane-summed scores, ties to the lower index, ascending."""
    return _largest_k(planes_score(planes), K)


def _largest_k(score: np.ndarray, K: int) -> np.ndarray:
    B, L = score.shape
    if not 0 <= K <= L:
        raise ValueError("need 0 <= K <= L")
    out = np.empty((B, K), dtype=np.int32)
    idx = np.arange(L)
    for b in range(B):
        order = np.lexsort((idx, -score[b].astype(np.float64)))   # primary: score desc; then index asc
        out[b] = np.sort(order[:K])
    return out
