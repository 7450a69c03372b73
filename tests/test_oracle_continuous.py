"""Pins for the continuous-reward grouping of the MDAP oracle (appendix on the grounding
task: o_i and o_j share an advantage group when |A_i - A_j| < eps, read as the connected
components of that relation) and for the traversal order of Alg. 1 (|A_i| descending)."""
import itertools

import numpy as np
import pytest

from oracle import group_advantage, prune_prompt, prune_batch, continuous_classes, visit_order
from oracle.mdap import class_kappa
from synth import CONFIGS, make_rollouts, continuous_rewards, plant_duplicates


def _components_brute(a, eps):
    """Connected components of the graph {(i, j): |a_i - a_j| < eps} by union-find over
    every pair, numbered by lowest member index."""
    G = len(a)
    parent = list(range(G))

    def find(x):
        while parent[x] != x:
            parent[x] = parent[parent[x]]
            x = parent[x]
        return x
    for i, j in itertools.combinations(range(G), 2):
        if abs(float(a[i]) - float(a[j])) < eps:
            parent[find(i)] = find(j)
    number, out = {}, []
    for i in range(G):
        r = find(i)
        number.setdefault(r, len(number))
        out.append(number[r])
    return out


@pytest.mark.parametrize("seed", range(40))
def test_single_linkage_equals_pairwise_components(seed):
    rng = np.random.default_rng(seed)
    G = int(rng.integers(1, 24))
    # values on a grid of ~eps spacing so that gaps fall on both sides of eps
    a = (rng.integers(0, 12, size=G) * rng.choice([0.5e-4, 0.9e-4, 1.1e-4, 3e-4])
         + rng.normal(0, 2e-5, size=G)).astype(np.float32)
    assert continuous_classes(a, 1e-4) == _components_brute(a, 1e-4)


def test_chain_is_one_group():
    # 0 ~ 0.6e-4 and 0.6e-4 ~ 1.2e-4 but |0 - 1.2e-4| >= eps: single linkage joins all three
    a = np.array([0.0, 0.6e-4, 1.2e-4, 5.0, 5.00005, -3.0], dtype=np.float32)
    assert continuous_classes(a, 1e-4) == [0, 0, 0, 1, 1, 2]
    assert _components_brute(a, 1e-4) == [0, 0, 0, 1, 1, 2]


def test_tiny_eps_reproduces_bit_equal_classes():
    ro = make_rollouts(CONFIGS[3], Q=16)
    adv, cls, _ = group_advantage(ro.rewards, ro.group_off)
    a32 = adv.astype(np.float32)
    for q in range(16):
        a, b = int(ro.group_off[q]), int(ro.group_off[q + 1])
        assert continuous_classes(a32[a:b], 1e-300) == [int(x) for x in cls[a:b]]


def test_huge_eps_is_one_group_and_zero_gap_links():
    a = np.array([3.0, -2.0, 0.5, 0.5], dtype=np.float32)
    assert continuous_classes(a, np.inf) == [0, 0, 0, 0]
    assert continuous_classes(a, 1e-300) == [0, 1, 2, 2]


def test_visit_order_is_abs_desc_then_index():
    a = np.array([0.5, -1.0, 1.0, 0.25, -0.5], dtype=np.float32)
    assert visit_order(5, a) == [1, 2, 0, 4, 3]
    assert visit_order(5) == [0, 1, 2, 3, 4]


def test_order_decides_which_near_tie_is_kept():
    # one continuous group {0, 1} (|A_0 - A_1| < eps) with identical token sequences
    # (theta = 0 < tau): Alg. 1 visits the larger |A| first and keeps it
    toks = [[1, 2, 3, 4], [1, 2, 3, 4], [9, 9, 9]]
    r = [0.70000, 0.70001, 0.1]
    adv, _, _ = group_advantage(np.asarray(r, np.float32), [0, 3])
    a32 = adv.astype(np.float32)
    assert abs(float(a32[0]) - float(a32[1])) < 1e-4 and abs(a32[1]) > abs(a32[0])
    keep, cnt, cls = prune_prompt(toks, r, [0, 1, 2], 1, 4, 5, 0.0, adv_q=a32, group_eps=1e-4)
    assert cls == [0, 0, 1] and keep == [False, True, True] and cnt == 2
    # index order (no advantages given) would keep member 0 of the same group instead
    keep_idx, _, _ = prune_prompt(toks, r, [0, 0, 1], 1, 4, 5, 0.0)
    assert keep_idx == [True, False, True]


def test_budget_kappa_from_first_visited_member():
    r = [0.70000, 0.70001, 0.1, 0.4]
    cls = [0, 0, 1, 2]
    a32 = group_advantage(np.asarray(r, np.float32), [0, 4])[0].astype(np.float32)
    order = visit_order(4, a32)
    kap = class_kappa(r, cls, order)
    s = sum(r)
    assert kap[0] == abs(4 * r[1] - s)  # member 1 has the larger |A|
    assert kap[1] == abs(4 * r[2] - s) and kap[2] == abs(4 * r[3] - s)


def test_batch_continuous_matches_per_question_groups():
    cfg = CONFIGS[5]
    ro = plant_duplicates(make_rollouts(cfg, Q=12, len_range=(16, 64), V=4096))
    rw = continuous_rewards(ro.group_off, seed=5)
    adv, cls, valid = group_advantage(rw, ro.group_off)
    a32 = adv.astype(np.float32)
    keep, cnt, used = prune_batch(ro.token_ids, ro.traj_tok_off, rw, ro.group_off, cls, valid,
                                  keep_ratio=0.4, adv=a32, group_eps=1e-4, return_classes=True)
    linked = 0
    for q in range(12):
        a, b = int(ro.group_off[q]), int(ro.group_off[q + 1])
        assert list(used[a:b]) == _components_brute(a32[a:b], 1e-4)
        linked += len(set(used[a:b])) < len(set(rw[a:b]))
        G = b - a
        assert keep[a:b].sum() == max(1, min(G, int(np.floor(0.4 * G + 0.5))))
    # the recipe really produces near-ties that merge distinct rewards into one group
    assert linked > 0


def test_gap_equal_to_eps_splits_and_sign_matters():
    f = np.float32(1e-4)
    a = np.array([0.0, f], dtype=np.float32)
    assert continuous_classes(a, float(f)) == [0, 1]                   # |gap| < eps is strict
    assert continuous_classes(a, float(np.nextafter(float(f), np.inf))) == [0, 0]
    # groups are over signed advantages: +A and -A are far apart
    assert continuous_classes(np.array([0.5, -0.5], np.float32), 1e-4) == [0, 1]
