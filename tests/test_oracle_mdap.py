"""Pins for the oracle's MDAP pruning, budget and compaction (Sec. 3.2, Alg. 1
Phase 2): hand-derived fixtures, exact boundary cases, brute force over all subsets,
and an independent sort-key formulation of the budget."""
from fractions import Fraction
import itertools
import json
import os

import numpy as np
import pytest

from oracle import (ngram_set, jaccard_counts, theta_below_tau, greedy_mdap_class,
                    budget_keep, prune_prompt, prune_batch, compact, group_advantage)
from oracle.mdap import budget_size, class_kappa


def test_ngram_sets():
    assert ngram_set([5, 5, 7, 5], 1) == {(5,), (7,)}
    assert ngram_set([5, 5, 7, 5], 2) == {(5, 5), (5, 7), (7, 5)}
    assert ngram_set([5, 5, 7, 5], 3) == {(5, 5, 7), (5, 7, 5)}
    assert ngram_set([5, 5, 7, 5], 5) == set()
    assert ngram_set([], 1) == set()


def test_golden_jaccard(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "jaccard.json")))
    for c in d["cases"]:
        sa, sb = ngram_set(c["a"], c["n"]), ngram_set(c["b"], c["n"])
        inter, union = jaccard_counts(sa, sb)
        assert (inter, union) == (c["inter"], c["union"]), c
        theta = Fraction(union - inter, union) if union else Fraction(0)
        assert theta == Fraction(c["theta"])
        assert theta_below_tau(inter, union, 4, 5) == c["below_tau_4_5"]


def test_theta_equal_tau_not_pruned_where_float_would():
    # |inter|/|union| = 1/5 gives theta = 4/5 = tau exactly: strict '<' keeps it.
    assert not theta_below_tau(1, 5, 4, 5)
    # the float formulations that are easy to write get this wrong
    assert (1 / 5) > (1 - 0.8)
    assert (1 - 4 / 5) < 0.2
    for k in range(1, 50):
        assert not theta_below_tau(k, 5 * k, 4, 5)
        assert theta_below_tau(k + 1, 5 * k, 4, 5)


def test_golden_mdap_prompt(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "mdap_prompt.json")))
    for p in d["prompts"]:
        r = np.asarray(p["rewards"], dtype=np.float32)
        _, cls, _ = group_advantage(r, [0, len(r)])
        assert list(cls) == p["class_id"]
        keep, cnt, _ = prune_prompt(p["tokens"], list(map(float, r)), list(cls), 1, 4, 5, 0.0)
        assert [int(k) for k in keep] == p["mdap_keep"] and cnt == p["mdap_count"]
        for rho, want in p["budget"].items():
            keep, cnt, _ = prune_prompt(p["tokens"], list(map(float, r)), list(cls), 1, 4, 5,
                                        float(rho))
            assert [int(k) for k in keep] == want, (rho, keep)
            assert cnt == p["mdap_count"]


def _conflict(sets, i, j, tn, td):
    inter, union = jaccard_counts(sets[i], sets[j])
    return theta_below_tau(inter, union, tn, td)


def _all_mis(members, sets, tn, td):
    out = []
    for r in range(1, len(members) + 1):
        for sub in itertools.combinations(members, r):
            if any(_conflict(sets, a, b, tn, td) for a, b in itertools.combinations(sub, 2)):
                continue
            rest = [m for m in members if m not in sub]
            if all(any(_conflict(sets, m, s, tn, td) for s in sub) for m in rest):
                out.append(tuple(sorted(sub)))
    return out


def _planted_class(rng, size):
    base = [list(rng.integers(0, 12, size=rng.integers(3, 9))) for _ in range(3)]
    toks = []
    for _ in range(size):
        t = list(base[rng.integers(0, 3)])
        for _ in range(rng.integers(0, 3)):  # mutate a little
            t[rng.integers(0, len(t))] = int(rng.integers(0, 12))
        toks.append(t)
    return toks


@pytest.mark.parametrize("seed", range(40))
def test_greedy_is_lexicographically_first_mis(seed):
    rng = np.random.default_rng(seed)
    size = int(rng.integers(1, 9))
    toks = _planted_class(rng, size)
    n = int(rng.integers(1, 3))
    tn, td = [(4, 5), (1, 2), (3, 5), (9, 10)][seed % 4]
    sets = {i: ngram_set(t, n) for i, t in enumerate(toks)}
    members = list(range(size))
    kept = greedy_mdap_class(members, sets, tn, td)
    mis = _all_mis(members, sets, tn, td)
    assert tuple(kept) in mis
    assert tuple(kept) == min(mis)
    assert kept[0] == 0  # |S'_k| >= 1: the first member is always kept


def test_tau_special_cases():
    rng = np.random.default_rng(7)
    for _ in range(20):
        size = int(rng.integers(2, 9))
        toks = _planted_class(rng, size)
        sets = {i: ngram_set(t, 1) for i in range(size) for t in [toks[i]]}
        members = list(range(size))
        # tau = 0: nothing is pruned (GRPO)
        assert greedy_mdap_class(members, sets, 0, 1) == members
        # tau > 1: exactly one trajectory per class (advantage-only ablation)
        assert greedy_mdap_class(members, sets, 2, 1) == [0]
        # tau = 1: one per class when every pair shares an n-gram
        if all(sets[i] & sets[j] for i in members for j in members):
            assert greedy_mdap_class(members, sets, 1, 1) == [0]


def test_budget_sizes():
    assert [budget_size(G, 0.4) for G in (8, 12, 16)] == [3, 5, 6]
    assert [budget_size(G, 0.5) for G in (8, 12, 16)] == [4, 6, 8]
    assert budget_size(1, 0.5) == 1 and budget_size(3, 0.01) == 1
    assert budget_size(4, 1.0) == 4
    # exact halves round up (floor(x + 1/2)), not to even
    assert budget_size(5, 0.5) == 3 and budget_size(9, 0.5) == 5


def _budget_by_sort_key(rewards, cls, mdap, rho):
    """Independent formulation: member key = (tier, rank inside its class tier,
    position of its class); the K smallest keys are kept."""
    G = len(rewards)
    kap = class_kappa(rewards, cls)
    first = {}
    for i, c in enumerate(cls):
        first.setdefault(c, i)
    pos = {c: p for p, c in enumerate(sorted(kap, key=lambda c: (-kap[c], first[c])))}
    keys = []
    for i in range(G):
        tier = 0 if mdap[i] else 1
        rank = sum(1 for j in range(i) if cls[j] == cls[i] and bool(mdap[j]) == bool(mdap[i]))
        keys.append(((tier, rank, pos[cls[i]]), i))
    K = budget_size(G, rho)
    chosen = {i for _, i in sorted(keys)[:K]}
    return [i in chosen for i in range(G)]


@pytest.mark.parametrize("seed", range(60))
def test_budget_properties(seed):
    rng = np.random.default_rng(100 + seed)
    G = int(rng.choice([2, 3, 5, 8, 12, 16]))
    rewards = [float(x) for x in rng.choice([0.0, 1.0, 1.1, 0.1], size=G)]
    _, cls, _ = group_advantage(np.asarray(rewards, np.float32), [0, G])
    cls = list(cls)
    mdap = [bool(x) for x in rng.integers(0, 2, size=G)]
    for c in set(cls):  # MDAP always keeps the first member of a class
        mdap[cls.index(c)] = True
    rho = float(rng.choice([0.1, 0.25, 0.4, 0.5, 0.75, 1.0]))
    keep = budget_keep(rewards, cls, mdap, rho)
    K = budget_size(G, rho)
    assert sum(keep) == K
    ncls = len(set(cls))
    if K >= ncls:
        assert set(cls[i] for i in range(G) if keep[i]) == set(cls)
    if sum(mdap) <= K:
        assert all(keep[i] for i in range(G) if mdap[i])
    else:
        assert all(mdap[i] for i in range(G) if keep[i])
    assert keep == _budget_by_sort_key(rewards, cls, mdap, rho)


def test_budget_orders_minority_class_first():
    # binary rewards, 2 successes of 8: the success class has the larger |A|
    r = [1.0, 0.0, 0.0, 1.0, 0.0, 0.0, 0.0, 0.0]
    cls = [0, 1, 1, 0, 1, 1, 1, 1]
    keep = budget_keep(r, cls, [True] * 8, 0.25)  # K = 2
    assert keep == [True, True, False, False, False, False, False, False]
    keep = budget_keep(r, cls, [True] * 8, 0.5)  # K = 4: 0,1,3,2
    assert [i for i in range(8) if keep[i]] == [0, 1, 2, 3]


def test_prune_batch_and_compaction():
    rng = np.random.default_rng(3)
    sizes = [8, 8, 12]
    goff = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    N = goff[-1]
    lens = rng.integers(0, 6, size=N)
    toff = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    tok = rng.integers(0, 5, size=toff[-1]).astype(np.int32)
    r = rng.integers(0, 2, size=N).astype(np.float32)
    r[8:16] = 1.0  # all equal question
    _, cls, valid = group_advantage(r, goff, drop_uniform=True)
    keep, counts = prune_batch(tok, toff, r, goff, cls, valid, 1, 4, 5, 0.5)
    assert keep[8:16].sum() == 0 and counts[1] == 0
    kept, koff, src = compact(keep, toff)
    assert list(kept) == [i for i in range(N) if keep[i]]
    assert koff[0] == 0 and koff[-1] == len(src)
    for s, i in enumerate(kept):
        assert koff[s + 1] - koff[s] == lens[i]
        assert list(src[koff[s]:koff[s + 1]]) == list(range(toff[i], toff[i + 1]))
    # empty input
    k2, o2, s2 = compact(np.zeros(0, np.uint8), np.zeros(1, np.int64))
    assert len(k2) == 0 and list(o2) == [0] and len(s2) == 0
