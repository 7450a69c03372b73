"""Pins for the oracle's group-relative advantage (Sec. 3.2, Eq. advantage)."""
import json
import math
import os

import numpy as np

from oracle import group_advantage


def test_golden_binary_closed_form(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "advantage_binary.json")))
    for c in d["cases"]:
        r = np.asarray(c["rewards"], dtype=np.float32)
        adv, cls, valid = group_advantage(r, [0, len(r)], ddof=c["ddof"], eps=c["eps"])
        np.testing.assert_allclose(adv, c["adv"], rtol=1e-12, atol=1e-15)


def test_binary_formula_all_k():
    # std(ddof=1) of k ones among G: sqrt(k (G-k) / (G (G-1)))
    for G in (2, 8, 12, 16):
        for k in range(1, G):
            r = np.zeros(G, dtype=np.float32)
            r[:k] = 1
            adv, _, _ = group_advantage(r, [0, G], eps=0.0)
            s = math.sqrt(k * (G - k) / (G * (G - 1)))
            assert abs(adv[0] - (1 - k / G) / s) < 1e-12
            assert abs(adv[-1] - (-k / G) / s) < 1e-12


def test_sum_zero_and_numpy_std():
    rng = np.random.default_rng(1)
    sizes = rng.integers(2, 20, size=30)
    off = np.concatenate([[0], np.cumsum(sizes)])
    r = rng.normal(size=off[-1]).astype(np.float32)
    adv, cls, valid = group_advantage(r, off, ddof=1, eps=0.0)
    for q in range(len(sizes)):
        a, b = off[q], off[q + 1]
        rr = r[a:b].astype(np.float64)
        assert abs(adv[a:b].sum()) < 1e-12
        ref = (rr - rr.mean()) / np.std(rr, ddof=1)
        np.testing.assert_allclose(adv[a:b], ref, rtol=1e-12, atol=1e-13)
        # continuous rewards: every member is its own class
        assert len(set(cls[a:b])) == b - a
    # ddof = 0 variant against numpy as well
    adv0, _, _ = group_advantage(r, off, ddof=0, eps=0.0)
    rr = r[off[0]:off[1]].astype(np.float64)
    np.testing.assert_allclose(adv0[off[0]:off[1]], (rr - rr.mean()) / np.std(rr),
                               rtol=1e-12)


def test_classes_and_dapo_drop():
    r = np.asarray([1, 0, 1, 0.5, 0, 2, 2, 2], dtype=np.float32)
    adv, cls, valid = group_advantage(r, [0, 5, 8], drop_uniform=True)
    assert list(cls) == [0, 1, 0, 2, 1, 0, 0, 0]
    assert list(valid) == [1, 0]
    assert np.all(adv[5:] == 0.0)
    # equal reward <=> equal advantage inside a question with std > 0
    for i in range(5):
        for j in range(5):
            assert (cls[i] == cls[j]) == (adv[i] == adv[j])
    _, _, valid2 = group_advantage(r, [0, 5, 8], drop_uniform=False)
    assert list(valid2) == [1, 1]


def test_singleton_group():
    adv, cls, valid = group_advantage(np.asarray([3.0], np.float32), [0, 1])
    assert adv[0] == 0.0 and cls[0] == 0 and valid[0] == 1
