"""Pins of the oracle's Wanda mask selection (the weight update's input).

An entry is kept iff fewer than k entries of its row (or group of 4) beat it,
where a beats b when score(a) > score(b), or the scores are equal and a has
the lower index. The tests evaluate that definition by brute force.
"""
import numpy as np
import pytest

import oracle
import workloads


def _brute(score, keep):
    n = len(score)
    out = np.zeros(n, dtype=np.uint8)
    for a in range(n):
        beats = sum(1 for b in range(n)
                    if score[b] > score[a] or (score[b] == score[a] and b < a))
        out[a] = beats < keep
    return out


def _scores(W, c):
    # Squared saliency, written out element by element.
    n, d = W.shape
    out = np.empty((n, d))
    for j in range(n):
        for i in range(d):
            w = float(W[j, i])
            out[j, i] = (w * w) * float(c[i])
    return out


@pytest.mark.parametrize("sparsity", [0.0, 0.3, 0.5, 0.6, 0.99, 1.0])
def test_unstructured_against_brute_force(sparsity):
    rng = np.random.default_rng(7)
    n, d = 6, 23
    # Few distinct magnitudes: many exact ties.
    W = (rng.integers(-3, 4, (n, d)) * 0.25).astype(np.float32)
    c = rng.choice([1.0, 4.0, 0.25], d).astype(np.float32)
    m = oracle.wanda_mask(W, c, "unstructured", sparsity)
    keep = d - int(np.floor(sparsity * d))
    assert np.all(m.sum(axis=1) == keep)
    s = _scores(W, c)
    for j in range(n):
        np.testing.assert_array_equal(m[j], _brute(s[j], keep))


def test_2to4_against_brute_force_and_hand_ties():
    rng = np.random.default_rng(8)
    W = (rng.integers(-2, 3, (5, 32)) * 0.5).astype(np.float32)
    c = np.ones(32, dtype=np.float32)
    m = oracle.wanda_mask(W, c, "2:4")
    s = _scores(W, c)
    for j in range(5):
        for g in range(0, 32, 4):
            np.testing.assert_array_equal(m[j, g:g + 4], _brute(s[j, g:g + 4], 2))
    # All four equal: the first two are kept; zeros are never preferred.
    W = np.array([[1, 1, 1, 1, 0, 2, 0, 0, -3, 3, 3, 1]], dtype=np.float32)
    m = oracle.wanda_mask(W, np.ones(12, np.float32), "2:4")
    np.testing.assert_array_equal(m[0], [1, 1, 0, 0, 1, 1, 0, 0, 1, 1, 0, 0])
    # The column norm decides between equal weights.
    W = np.array([[1, 1, 1, 1]], dtype=np.float32)
    c = np.array([1, 9, 4, 9], dtype=np.float32)
    np.testing.assert_array_equal(oracle.wanda_mask(W, c, "2:4")[0], [0, 1, 0, 1])
    # NaN scores rank last, -0 equals +0, a larger weight of either sign wins.
    W = np.array([[np.nan, 0.0, -0.0, 2.0, -3.0, np.nan, 1.0, 0.5]], dtype=np.float32)
    np.testing.assert_array_equal(oracle.wanda_mask(W, np.ones(8, np.float32), "2:4")[0],
                                  [0, 1, 0, 1, 1, 0, 1, 0])


def test_matches_the_host_generator_on_a_layer():
    cfg = workloads.GPT2_FC.with_tokens(4096).with_cols(64)
    X = workloads.x_all(cfg)
    W0 = workloads.w0(cfg)
    cs = workloads.col_sq_norms(cfg, X)
    np.testing.assert_array_equal(oracle.wanda_mask(W0, cs, "unstructured", 0.5),
                                  workloads.wanda_unstructured(W0, cs, 0.5))
    np.testing.assert_array_equal(oracle.wanda_mask(W0, cs, "2:4"),
                                  workloads.wanda_2to4(W0, cs))
