"""Pins for the DP-alignment fill of Alg. 1 (kept count up to a multiple of d by adding the
highest-|A| unselected trajectories round-robin over the questions)."""
import numpy as np
import pytest

from oracle import dp_align_fill


def _fill_by_keys(keep, adv, group_off, valid, d):
    """Second formulation: rank every unselected trajectory inside its question by
    (|A| descending, index); the round-robin takes candidates in (rank, question) order,
    so the fill is the first `need` candidates of that order."""
    keep = np.array(keep, dtype=np.uint8)
    a = np.abs(np.asarray(adv, np.float32).astype(np.float64))
    cands = []
    for q in range(len(group_off) - 1):
        if valid is not None and not valid[q]:
            continue
        un = [i for i in range(group_off[q], group_off[q + 1]) if not keep[i]]
        un.sort(key=lambda i: (-a[i], i))
        cands += [(r, q, i) for r, i in enumerate(un)]
    cands.sort()
    need = (-int(keep.sum())) % d
    for _, _, i in cands[:need]:
        keep[i] = 1
    return keep


def test_hand_example():
    # two questions of 4; kept {0, 4, 5} -> 3 kept, d = 4 -> one more: question 0's best
    adv = np.array([0.9, -0.2, 0.5, -1.5, 0.3, 0.1, -0.7, 0.7], np.float32)
    keep = np.array([1, 0, 0, 0, 1, 1, 0, 0], np.uint8)
    k, n = dp_align_fill(keep, adv, [0, 4, 8], None, 4)
    assert n == 1 and list(k) == [1, 0, 0, 1, 1, 1, 0, 0]
    # d = 8: need 5 -> round 0: q0 -> 3, q1 -> 6 (|-0.7| ties |0.7|: lower index); round 1:
    # q0 -> 2, q1 -> 7; round 2: q0 -> 1
    k, n = dp_align_fill(keep, adv, [0, 4, 8], None, 8)
    assert n == 5 and list(k) == [1, 1, 1, 1, 1, 1, 1, 1]
    k, n = dp_align_fill(keep, adv, [0, 4, 8], None, 7)
    assert n == 4 and list(k) == [1, 0, 1, 1, 1, 1, 1, 1]


def test_aligned_and_trivial_cases_unchanged():
    adv = np.linspace(-1, 1, 12).astype(np.float32)
    keep = np.array([1] * 6 + [0] * 6, np.uint8)
    for d in (1, 2, 3, 6):
        k, n = dp_align_fill(keep, adv, [0, 6, 12], None, d)
        assert n == 0 and np.array_equal(k, keep)


def test_not_enough_candidates_stops():
    adv = np.ones(5, np.float32)
    keep = np.array([1, 1, 1, 0, 0], np.uint8)
    k, n = dp_align_fill(keep, adv, [0, 5], None, 8)
    assert n == 2 and k.sum() == 5
    # invalid questions never contribute
    k, n = dp_align_fill(keep, adv, [0, 5], [0], 4)
    assert n == 0 and k.sum() == 3


@pytest.mark.parametrize("seed", range(30))
def test_matches_rank_question_order(seed):
    rng = np.random.default_rng(seed)
    Q = int(rng.integers(1, 9))
    sizes = rng.integers(1, 9, size=Q)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    N = int(off[-1])
    adv = rng.choice([-1.0, -0.5, 0.0, 0.5, 1.0, 0.25], size=N).astype(np.float32)
    keep = (rng.uniform(size=N) < 0.4).astype(np.uint8)
    valid = (rng.uniform(size=Q) < 0.85).astype(np.uint8)
    for i in range(Q):
        if not valid[i]:
            keep[off[i]:off[i + 1]] = 0
    d = int(rng.integers(2, 9))
    k, n = dp_align_fill(keep, adv, off, valid, d)
    assert np.array_equal(k, _fill_by_keys(keep, adv, off, valid, d))
    assert n == int(k.sum() - keep.sum())
    total = sum(int(off[i + 1] - off[i]) for i in range(Q) if valid[i])
    if total >= keep.sum() + (-int(keep.sum())) % d:
        assert k.sum() % d == 0
