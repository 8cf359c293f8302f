"""Pins of the oracle's per-position statistics against closed forms and library routines."""
import math

import numpy as np
import pytest
import scipy.special
import scipy.stats

from oracle.stats import softmax_stats, entropy_from_logits, confidence

V = 97
MASK = V - 1


def _masked(logits):
    logits = np.array(logits, dtype=np.float64)
    logits[:, MASK] = -np.inf
    return logits


def test_one_hot_has_zero_entropy():
    l = np.full((1, V), -np.inf)
    l[0, 17] = 3.0
    st = softmax_stats(l, 4)
    assert st.H[0] == 0.0
    assert st.argmax[0] == 17
    assert confidence(st)[0] == 1.0


def test_uniform_entropy_is_log_of_support():
    # [MASK] excluded: uniform over V-1 tokens
    st = softmax_stats(_masked(np.zeros((2, V))), 5)
    assert np.allclose(st.H, math.log(V - 1), rtol=0, atol=1e-12)
    # ties resolve to the lowest token ids
    assert st.argmax.tolist() == [0, 0]
    assert st.topk_id[0].tolist() == [0, 1, 2, 3, 4]
    assert np.allclose(confidence(st), 1.0 / (V - 1))


def test_two_point_distribution_is_binary_entropy():
    for q in (0.5, 0.7, 0.9, 0.99):
        l = np.full((1, V), -np.inf)
        l[0, 3] = math.log(q)
        l[0, 40] = math.log(1 - q)
        h = -q * math.log(q) - (1 - q) * math.log(1 - q)
        st = softmax_stats(l, 2)
        assert abs(st.H[0] - h) < 1e-12
        assert st.topk_id[0].tolist() == ([3, 40] if q > 0.5 else [3, 40])


def test_entropy_matches_scipy():
    rng = np.random.default_rng(0)
    l = _masked(rng.normal(0, 3.0, (16, V)))
    p = scipy.special.softmax(l, axis=1)
    assert np.allclose(entropy_from_logits(l), scipy.stats.entropy(p, axis=1), atol=1e-12)
    st = softmax_stats(l, 8)
    assert np.allclose(st.lse, scipy.special.logsumexp(l, axis=1), atol=1e-12)


def test_shift_invariance():
    rng = np.random.default_rng(1)
    l = _masked(rng.normal(0, 2.0, (8, V)))
    a, b = softmax_stats(l, 6), softmax_stats(l + 123.25, 6)
    assert np.allclose(a.H, b.H, atol=1e-10)
    assert np.array_equal(a.topk_id, b.topk_id)
    assert np.allclose(a.lse + 123.25, b.lse)
    assert np.allclose(a.lmax + 123.25, b.lmax)


def test_topk_brute_force_with_ties():
    rng = np.random.default_rng(2)
    l = _masked(rng.integers(-3, 4, (20, V)).astype(np.float64))   # many exact ties
    K = 7
    st = softmax_stats(l, K)
    for r in range(l.shape[0]):
        ref = sorted(range(V), key=lambda v: (-l[r, v], v))[:K]
        assert st.topk_id[r].tolist() == ref
        assert st.argmax[r] == ref[0]
        assert np.array_equal(st.topk_logit[r], l[r, ref])


def test_vocab_permutation_equivariance():
    rng = np.random.default_rng(3)
    l = rng.normal(0, 1.0, (4, V))
    perm = rng.permutation(V)
    a = softmax_stats(l, 5)
    b = softmax_stats(l[:, perm], 5)
    assert np.allclose(a.H, b.H)
    assert np.array_equal(a.topk_id, perm[b.topk_id])


def test_margins():
    l = np.array([[5.0, 4.0, 3.5, 1.0]])
    st = softmax_stats(l, 2)
    assert st.argmax_margin[0] == 1.0
    assert st.topk_margin[0] == 0.5
