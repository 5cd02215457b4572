"""Pins of the oracle's token selection (Sec. 3.2 "Random token selection",
App. A.4) and of the top-k variant."""
import numpy as np
import pytest
from scipy import stats

from oracle import select as sel
from oracle.numerics import f32_to_bf16_bits

pytestmark = pytest.mark.cpu


def test_splitmix64_published_stream():
    # SplitMix64 reference output for initial state 1234567 (Steele, Lea, Flood 2014;
    # the values printed by the authors' reference C code).
    want = [6457827717110365317, 3203168211198807973, 9817491932198370423,
            4593380528125082431, 16408922859458223821]
    assert [int(v) for v in sel.splitmix64_stream(1234567, 5)] == want


@pytest.mark.parametrize("B,L,K", [(1, 128, 32), (3, 100, 25), (2, 17, 1), (1, 16200, 4050), (2, 9, 9), (2, 9, 0)])
def test_random_invariants(B, L, K):
    idx = sel.select_random(B, L, K, seed=42, step=3)
    assert idx.shape == (B, K) and idx.dtype == np.int32
    if K:
        assert (idx >= 0).all() and (idx < L).all()
        assert (np.diff(idx, axis=1) > 0).all()          # strictly increasing => no repeats
    if K == L:
        assert (idx == np.arange(L)).all()


def test_random_fresh_draws_and_determinism():
    a = sel.select_random(2, 256, 64, seed=42, step=0)
    assert np.array_equal(a, sel.select_random(2, 256, 64, seed=42, step=0))
    assert not np.array_equal(a, sel.select_random(2, 256, 64, seed=42, step=1))
    assert not np.array_equal(a, sel.select_random(2, 256, 64, seed=43, step=0))
    assert not np.array_equal(a[0], a[1])                 # samples draw independently


def test_random_inclusion_uniform():
    # Uniform without replacement: every token is kept with probability K/L.
    L, K, n = 64, 16, 4000
    counts = np.zeros(L)
    pair = 0
    for s in range(n):
        idx = sel.select_random(1, L, K, seed=7, step=s)[0]
        counts[idx] += 1
        pair += (0 in idx) and (1 in idx)
    _, p = stats.chisquare(counts)
    assert p > 1e-4, p
    # pairwise inclusion probability K(K-1)/(L(L-1)) (sampling without replacement)
    want = K * (K - 1) / (L * (L - 1))
    assert abs(pair / n - want) < 5 * np.sqrt(want * (1 - want) / n)


def test_random_rank_of_first_uniform():
    # The smallest key's token is uniform over 0..L-1 (first entry of a uniform permutation).
    L, n = 32, 6000
    first = [int(np.argmin(sel.random_keys(L, 0, 11, s))) for s in range(n)]
    counts = np.bincount(first, minlength=L)
    _, p = stats.chisquare(counts)
    assert p > 1e-4, p


# ------------------------------------------------------------------------- top-k

def _bf16(a):
    return f32_to_bf16_bits(np.asarray(a, dtype=np.float32))


def test_topk_score_within_fp32_bound():
    rng = np.random.default_rng(1)
    B, L, D = 2, 50, 1024
    xt = _bf16(rng.standard_normal((B, L, D)))
    xp = _bf16(rng.standard_normal((B, L, D)))
    s = sel.topk_score(xt, xp).astype(np.float64)
    from oracle.numerics import bf16_bits_to_f32
    exact = ((bf16_bits_to_f32(xt).astype(np.float64) - bf16_bits_to_f32(xp)) ** 2).sum(-1)
    # each term carries <= 2 roundings (difference, square), the tree depth is <= 16 + 6 additions
    u = 2.0 ** -24
    assert (np.abs(s - exact) <= (2 + 16 + 6) * u * exact * 1.01).all()


def test_topk_score_evaluation_order_hand_case():
    # D = 512 bf16: 64 chunks, one per lane.  Lane 0 holds a single 1.0, lanes 1..63 a
    # single 2^-26.  Left-to-right summation stays at 1.0 and the exact sum rounds to
    # 1 + 8u (u = 2^-23); the butterfly gives 1 + 7u (see the module header).
    D = 512
    xt = np.zeros((1, 1, D), dtype=np.float32)
    xt[0, 0, 0] = 1.0
    for lane in range(1, 64):
        xt[0, 0, lane * 8] = 2.0 ** -13
    s = sel.topk_score(_bf16(xt), _bf16(np.zeros_like(xt)))
    assert s[0, 0] == np.float32(1.0 + 7 * 2.0 ** -23)


def test_topk_matches_fp64_bruteforce_when_no_near_ties():
    rng = np.random.default_rng(2)
    B, L, D, K = 2, 300, 64, 75
    xt = _bf16(rng.standard_normal((B, L, D)))
    xp = _bf16(rng.standard_normal((B, L, D)))
    from oracle.numerics import bf16_bits_to_f32
    exact = ((bf16_bits_to_f32(xt).astype(np.float64) - bf16_bits_to_f32(xp)) ** 2).sum(-1)
    idx = sel.select_topk(xt, xp, K)
    for b in range(B):
        srt = np.sort(exact[b])[::-1]
        assert (srt[K - 1] - srt[K]) / srt[K - 1] > 1e-5      # no near-tie at the boundary
        want = np.sort(np.argsort(-exact[b], kind="stable")[:K])
        assert np.array_equal(idx[b], want)


def test_topk_ties_go_to_lower_index():
    B, L, D, K = 1, 10, 16, 4
    xt = np.zeros((B, L, D), dtype=np.float32)
    xt[0, [2, 5, 7, 8], 0] = 1.0       # four equal scores...
    xt[0, 9, 0] = 2.0                  # ...and one larger
    idx = sel.select_topk(_bf16(xt), _bf16(np.zeros_like(xt)), K)
    assert idx.tolist() == [[2, 5, 7, 9]]
    idx = sel.select_topk(_bf16(xt), _bf16(np.zeros_like(xt)), L)
    assert idx.tolist() == [list(range(L))]
    zero = sel.select_topk(_bf16(np.zeros_like(xt)), _bf16(np.zeros_like(xt)), 3)
    assert zero.tolist() == [[0, 1, 2]]
