"""Pins of the oracle's attention-score selector (Sec. 4.4 "Random vs. learned token
selection"; Tab. selection): per-head column sums of the attention probabilities and the
top-K over plane-summed fp32 scores."""
import math

import numpy as np
import pytest

from oracle import select

pytestmark = pytest.mark.cpu


def _qk(B=2, H=3, S=17, hd=8, seed=0):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((B, H, S, hd)), rng.standard_normal((B, H, S, hd))


def test_columns_add_up_to_rows():
    # every row of softmax sums to 1, so the S column sums of a head add up to S
    q, k = _qk()
    c = select.attention_colsums(q, k)
    assert np.allclose(c.sum(axis=2), q.shape[2], rtol=0, atol=1e-12)
    assert (c > 0).all()


def test_zero_queries_attend_uniformly():
    q, k = _qk()
    c = select.attention_colsums(np.zeros_like(q), k)
    assert np.allclose(c, 1.0, rtol=0, atol=1e-13)


def test_loop_written_softmax():
    q, k = _qk(B=1, H=2, S=5, hd=3, seed=4)
    c = select.attention_colsums(q, k)
    for h in range(2):
        want = [0.0] * 5
        for i in range(5):
            s = [sum(q[0, h, i, d] * k[0, h, j, d] for d in range(3)) / math.sqrt(3) for j in range(5)]
            e = [math.exp(x) for x in s]
            tot = sum(e)
            for j in range(5):
                want[j] += e[j] / tot
        assert np.allclose(c[0, h], want, rtol=1e-12, atol=0)


def test_token_permutation_permutes_scores():
    q, k = _qk(seed=7)
    perm = np.random.default_rng(1).permutation(q.shape[2])
    c = select.attention_colsums(q, k)
    cp = select.attention_colsums(q[:, :, perm], k[:, :, perm])
    assert np.allclose(cp, c[:, :, perm], rtol=1e-12, atol=1e-12)


def test_one_dominant_key_takes_the_attention():
    # a key aligned with every query and much longer than the others receives nearly all
    # attention: it is selected first
    q, k = _qk(B=1, H=1, S=9, hd=4, seed=3)
    q[:] = np.abs(q) + 0.5
    k[0, 0, 6] = 20.0
    c = select.attention_colsums(q, k)
    assert c[0, 0, 6] > 8.99
    idx = select.select_topk_planes(c.astype(np.float32), 1)
    assert idx.tolist() == [[6]]


def test_planes_sum_in_order_and_ties_go_low():
    # fp32 plane order: (1 + 2^-24) + 2^-24 rounds to 1 then to 1 (two half-ulp ties to even),
    # while the exact sum is 1 + 2^-23
    eps = np.float32(2.0 ** -24)
    planes = np.array([[[1.0, 1.0, 0.5], [eps, 0.0, 0.25], [eps, 0.0, 0.25]]], dtype=np.float32)
    s = select.planes_score(planes)
    assert s[0, 0] == np.float32(1.0) and s[0, 1] == np.float32(1.0)
    # tokens 0 and 1 tie at 1.0: K = 1 keeps the lower index; token 2 (1.0 as well) too
    assert select.select_topk_planes(planes, 1).tolist() == [[0]]
    assert select.select_topk_planes(planes, 2).tolist() == [[0, 1]]
    assert select.select_topk_planes(planes, 3).tolist() == [[0, 1, 2]]


def test_one_plane_is_plain_topk_ranking():
    rng = np.random.default_rng(5)
    sc = rng.random((3, 40)).astype(np.float32)
    got = select.select_topk_planes(sc[:, None, :], 11)
    for b in range(3):
        assert got[b].tolist() == sorted(np.argsort(-sc[b], kind="stable")[:11].tolist())
