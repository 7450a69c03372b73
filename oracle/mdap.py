"""Oracle: Maximizing Differential Advantage Pruning + stream compaction
(test infrastructure only; see oracle/__init__).

Paper, Sec. 3.2 and Alg. 1 Phase 2:
* partition a question's rollouts by advantage value (Eq. grouping);
* token n-gram Jaccard distance theta_ij = 1 - |N_n(o_i) & N_n(o_j)| / |N_n(o_i) | N_n(o_j)|
  where N_n(o) is the set of distinct contiguous n-grams of o's tokens;
* inside each class, traverse the members and keep o_i unless some already-kept
  o_j of the same class has theta_ij < tau (strict), i.e. a greedy maximal
  independent set of the conflict graph {theta < tau};
* the kept set of the question is the union over classes.

Readings where the paper is silent or ambiguous:
* traversal order inside a class: Alg. 1 orders by |A_i| descending, which is
  constant inside a bit-equal class, so ties are broken by ascending trajectory index;
* tau is a rational tau_num / tau_den and the comparison is done exactly
  (``fractions.Fraction``); theta of two empty n-gram sets is 0, and of one empty
  and one non-empty set is 1 (the definition with |union| > 0);
* keep-ratio budget (not in the paper; the workload fixes a keep ratio rho):
  K_q = clamp(floor(rho * G_q + 0.5), 1, G_q).  Classes are ordered by
  kappa_k = |G_q * r_k - sum_j r_j| descending (proportional to |A| of the class;
  the sum runs over the question's rewards in index order in float64), ties by
  lowest first member.  The priority list is a round-robin over the ordered
  classes taking each class's next MDAP-kept member (ascending index); once those
  run out, the round-robin continues over the MDAP-pruned members.  The first K_q
  entries are kept.  rho = 0 means pure MDAP.
* questions marked invalid (DAPO drop of all-equal groups) keep nothing and report
  an MDAP count of 0.

DP alignment (Alg. 1, after the union of the per-question sets): while the kept count
is not a multiple of the data-parallel divisor d, add the unselected trajectory with the
highest |A|, round-robin over the questions (``dp_align_fill``).

Continuous rewards (appendix on the grounding task; the only change the paper makes
for continuous rewards is to Eq. grouping): o_i and o_j share an advantage group
whenever |A_i - A_j| < eps (eps = 1e-4 there).  Readings:
* that relation is not transitive; the groups are its connected components (single
  linkage): sort a question's advantages, and a new group starts wherever the gap to
  the previous sorted value is >= eps;
* the advantages compared are the float32 values the advantage step outputs, read as
  exact float64, the gap computed in float64;
* groups are numbered by their lowest member index, like the bit-equal classes;
* members of a group now differ in |A|, so Alg. 1's traversal order (|A_i|
  descending) matters: members are visited by |A| descending, ties by index.  The
  budget follows the same order: a group's kappa is that of its first visited member,
  and each round-robin takes the group's next member in visiting order.  With
  bit-equal classes this is exactly the index order above.
"""
from fractions import Fraction
import math

import numpy as np


def ngram_set(tokens, n):
    """N_n(o): the set of distinct contiguous n-grams (as tuples) of a token list."""
    toks = [int(t) for t in tokens]
    return {tuple(toks[i:i + n]) for i in range(len(toks) - n + 1)}


def jaccard_counts(si, sj):
    """(|si & sj|, |si | sj|) of two n-gram sets."""
    inter = len(si & sj)
    return inter, len(si) + len(sj) - inter


def theta_below_tau(inter, union, tau_num, tau_den):
    """theta < tau, exactly, with theta = 1 - inter/union (0 when union == 0)."""
    theta = Fraction(union - inter, union) if union > 0 else Fraction(0)
    return theta < Fraction(tau_num, tau_den)


def greedy_mdap_class(members, sets, tau_num, tau_den):
    """S'_k: traverse ``members`` (in the given order) and keep o_i unless some kept
    o_j has theta_ij < tau.  ``sets`` maps member -> n-gram set."""
    kept = []
    for i in members:
        conflict = False
        for j in kept:
            inter, union = jaccard_counts(sets[i], sets[j])
            if theta_below_tau(inter, union, tau_num, tau_den):
                conflict = True
                break
        if not conflict:
            kept.append(i)
    return kept


def continuous_classes(adv_q, eps):
    """Groups of one question under |A_i - A_j| < eps (connected components, i.e.
    single linkage over the sorted advantages), numbered by lowest member index.
    ``adv_q``: the question's float32 advantages."""
    a = [float(np.float32(x)) for x in adv_q]
    G = len(a)
    srt = sorted(range(G), key=lambda i: (a[i], i))
    comp = [0] * G
    c = 0
    for p in range(1, G):
        if a[srt[p]] - a[srt[p - 1]] >= eps:
            c += 1
        comp[srt[p]] = c
    number = {}
    cls = []
    for i in range(G):
        number.setdefault(comp[i], len(number))
        cls.append(number[comp[i]])
    return cls


def visit_order(G, adv_q=None):
    """Traversal order of a question's members: |A| descending, ties by index (Alg. 1);
    ascending index when no advantages are given."""
    if adv_q is None:
        return list(range(G))
    a = [abs(float(np.float32(x))) for x in adv_q]
    return sorted(range(G), key=lambda i: (-a[i], i))


def class_kappa(rewards_q, cls_q, order=None):
    """kappa per class id: |G * r_k - sum_j r_j| in float64, sum in index order, r_k
    the reward of the class's first member in ``order`` (default: index order)."""
    G = len(rewards_q)
    s = 0.0
    for r in rewards_q:
        s += float(r)
    kap = {}
    for i in (order if order is not None else range(G)):
        c = cls_q[i]
        if c not in kap:
            kap[c] = abs(float(G) * float(rewards_q[i]) - s)
    return kap


def budget_size(G, keep_ratio):
    """K_q = clamp(floor(rho * G + 0.5), 1, G) in float64."""
    k = int(math.floor(float(keep_ratio) * float(G) + 0.5))
    return max(1, min(G, k))


def budget_keep(rewards_q, cls_q, mdap_keep_q, keep_ratio, order=None):
    """Apply the keep-ratio budget to one question.  Returns a bool list.
    ``order``: the members' visiting order (default: ascending index)."""
    G = len(rewards_q)
    order = list(order) if order is not None else list(range(G))
    kap = class_kappa(rewards_q, cls_q, order)
    first = {}
    for i, c in enumerate(cls_q):
        first.setdefault(c, i)
    corder = sorted(kap.keys(), key=lambda c: (-kap[c], first[c]))
    priority = []
    for tier in (True, False):
        lists = [[i for i in order if cls_q[i] == c and bool(mdap_keep_q[i]) == tier]
                 for c in corder]
        rnd = 0
        while any(rnd < len(l) for l in lists):
            for l in lists:
                if rnd < len(l):
                    priority.append(l[rnd])
            rnd += 1
    K = budget_size(G, keep_ratio)
    keep = [False] * G
    for i in priority[:K]:
        keep[i] = True
    return keep


def prune_prompt(tokens_q, rewards_q, cls_q, ngram_n, tau_num, tau_den, keep_ratio,
                 valid=True, adv_q=None, group_eps=0.0):
    """One question.  Returns (keep bool[G], mdap_count, classes used).
    ``adv_q`` (float32 advantages) sets the visiting order; with ``group_eps`` > 0 the
    classes are the continuous-reward groups of ``adv_q`` and ``cls_q`` is ignored."""
    G = len(rewards_q)
    if group_eps > 0:
        cls_q = continuous_classes(adv_q, group_eps)
    if not valid:
        return [False] * G, 0, cls_q
    order = visit_order(G, adv_q)
    sets = [ngram_set(t, ngram_n) for t in tokens_q]
    mdap = [False] * G
    for c in sorted(set(cls_q)):
        members = [i for i in order if cls_q[i] == c]
        for i in greedy_mdap_class(members, sets, tau_num, tau_den):
            mdap[i] = True
    count = sum(mdap)
    if keep_ratio > 0:
        return budget_keep(rewards_q, cls_q, mdap, keep_ratio, order), count, cls_q
    return mdap, count, cls_q


def prune_batch(token_ids, traj_tok_off, rewards, group_off, class_id, group_valid,
                ngram_n=1, tau_num=4, tau_den=5, keep_ratio=0.0, adv=None, group_eps=0.0,
                return_classes=False):
    """Whole batch.  Returns (keep_mask uint8[N], mdap_count int32[Q]) and, with
    ``return_classes``, the class ids used (int32[N]).  ``adv``: float32[N] advantages
    (visiting order; required when ``group_eps`` > 0)."""
    tok = np.asarray(token_ids)
    toff = np.asarray(traj_tok_off, dtype=np.int64)
    r32 = np.asarray(rewards, dtype=np.float32)
    goff = np.asarray(group_off, dtype=np.int64)
    Q = len(goff) - 1
    N = int(goff[-1])
    keep = np.zeros(N, dtype=np.uint8)
    counts = np.zeros(Q, dtype=np.int32)
    used = np.zeros(N, dtype=np.int32)
    if group_eps > 0 and adv is None:
        raise ValueError("continuous-reward groups need the advantages")
    for q in range(Q):
        a, b = int(goff[q]), int(goff[q + 1])
        toks = [tok[toff[i]:toff[i + 1]] for i in range(a, b)]
        cq = [int(x) for x in class_id[a:b]] if class_id is not None else [0] * (b - a)
        k, c, cl = prune_prompt(toks, [float(x) for x in r32[a:b]], cq, ngram_n, tau_num,
                                tau_den, keep_ratio, bool(group_valid[q]),
                                None if adv is None else np.asarray(adv[a:b], np.float32),
                                group_eps)
        keep[a:b] = np.asarray(k, dtype=np.uint8)
        counts[q] = c
        used[a:b] = np.asarray(cl, dtype=np.int32)
    if return_classes:
        return keep, counts, used
    return keep, counts


def dp_align_fill(keep_mask, adv, group_off, group_valid, d):
    """Alg. 1 DP alignment: while |S| mod d != 0, add an unselected trajectory with the
    highest |A|, round-robin over the questions.  Readings: one round visits the valid
    questions in index order and adds each one's best remaining unselected trajectory
    (|A| descending, float32 values, ties by lowest index); rounds repeat until |S| is a
    multiple of d or no unselected trajectory is left.  Returns (keep uint8[N], added)."""
    keep = np.array(keep_mask, dtype=np.uint8)
    d = int(d)
    if d <= 1:
        return keep, 0
    a = np.abs(np.asarray(adv, dtype=np.float32).astype(np.float64))
    off = np.asarray(group_off, dtype=np.int64)
    Q = len(off) - 1
    pools = []
    for q in range(Q):
        if group_valid is not None and not group_valid[q]:
            pools.append([])
            continue
        cand = [i for i in range(int(off[q]), int(off[q + 1])) if not keep[i]]
        pools.append(sorted(cand, key=lambda i: (-a[i], i)))
    added = 0
    while int(keep.sum()) % d != 0:
        progressed = False
        for q in range(Q):
            if int(keep.sum()) % d == 0:
                break
            if pools[q]:
                keep[pools[q].pop(0)] = 1
                added += 1
                progressed = True
        if not progressed:
            break
    return keep, added


def compact(keep_mask, traj_tok_off):
    """Stream compaction of kept trajectories (ascending index).

    Returns (kept_traj int32[Nk], kept_tok_off int64[Nk+1], tok_src int64[Tk]):
    kept token t of the compacted stream comes from source token tok_src[t].
    """
    keep = np.asarray(keep_mask).astype(bool)
    toff = np.asarray(traj_tok_off, dtype=np.int64)
    kept = [i for i in range(len(keep)) if keep[i]]
    off = [0]
    src = []
    for i in kept:
        a, b = int(toff[i]), int(toff[i + 1])
        src.extend(range(a, b))
        off.append(off[-1] + (b - a))
    return (np.asarray(kept, dtype=np.int32), np.asarray(off, dtype=np.int64),
            np.asarray(src, dtype=np.int64))
