"""Pins for the oracle's per-token policy entropy H_t = -sum_v p log p."""
import math

import numpy as np
import scipy.stats

import oracle


def test_uniform_softmax_is_log_v():
    V, d = 1000, 16
    H = np.random.default_rng(0).normal(size=(5, d))
    ent = oracle.token_entropy(H, np.zeros((V, d)))
    assert np.abs(ent - math.log(V)).max() < 1e-12


def test_two_class_closed_form():
    rng = np.random.default_rng(1)
    for _ in range(20):
        a, b = rng.normal(size=2) * 3
        # z = H W^T with H = [1], W = [[a], [b]]
        ent = oracle.token_entropy(np.ones((1, 1)), np.array([[a], [b]]))[0]
        p = 1.0 / (1.0 + math.exp(b - a))
        want = -p * math.log(p) - (1 - p) * math.log(1 - p)
        assert abs(ent - want) < 1e-12


def test_matches_scipy_entropy_and_is_shift_invariant():
    rng = np.random.default_rng(2)
    H = rng.normal(size=(7, 12))
    W = 0.7 * rng.normal(size=(50, 12))
    ent = oracle.token_entropy(H, W)
    z = H @ W.T
    for t in range(7):
        p = np.exp(z[t] - z[t].max())
        assert abs(ent[t] - scipy.stats.entropy(p / p.sum())) < 1e-12
    # adding a constant to every logit of a token (an extra unit feature) changes nothing
    H2 = np.concatenate([H, np.full((7, 1), 5.0)], axis=1)
    W2 = np.concatenate([W, np.ones((50, 1))], axis=1)
    assert np.abs(oracle.token_entropy(H2, W2) - ent).max() < 1e-11


def test_peaked_softmax_tends_to_zero():
    W = np.zeros((100, 1))
    W[7, 0] = 1.0
    ent = oracle.token_entropy(np.array([[800.0]]), W)[0]   # p_7 = 1 - ~1e-345
    assert 0.0 <= ent < 1e-300
