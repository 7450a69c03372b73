"""The slab plan of fastrl_policy_loss_fwd_bwd (host only, through the C ABI): slabs hold
whole sequences in order, at least one token each, never more than max(1.25 cap, longest
sequence) tokens, and the default slab does not grow with the token count, so the
exp-logit buffer [slab, V] stays bounded whatever T is."""
import ctypes

import numpy as np
import pytest

from synth import CONFIGS, make_rollouts


@pytest.fixture(scope="module")
def fr():
    import paper_2609_36932_amd as m
    return m


def _args(fr, lengths, cap):
    off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    a = fr.LossArgs()
    dummy = ctypes.c_void_p(256)
    a.dtype, a.d, a.V, a.S, a.T = fr.BF16, 3584, 152064, len(lengths), int(off[-1])
    a.hidden = a.W = a.token_ids = a.old_logp = a.seq_off = a.loss = a.adv = dummy
    a.seq_off_host = ctypes.c_void_p(off.ctypes.data)
    a.eps_low, a.eps_high = 0.2, 0.2
    a.slab_tokens = cap
    return a, off


def _check(fr, lengths, cap):
    a, off = _args(fr, np.asarray(lengths, dtype=np.int64), cap)
    begin, tc_max = fr.slab_plan(a)
    S = len(lengths)
    capv = cap if cap > 0 else 32768
    assert begin[0] == 0 and begin[-1] == S and all(np.diff(begin) > 0)
    sizes = np.diff(off[np.asarray(begin)])
    assert tc_max == (sizes.max() if len(sizes) else 0)
    longest = max(lengths) if S else 0
    assert tc_max <= max(capv + capv // 4, longest), (tc_max, capv, longest)
    if off[-1] > 0:
        assert np.all(sizes > 0)
    return begin, sizes


def test_long_sequences_do_not_pile_into_the_last_slab(fr):
    rng = np.random.default_rng(0)
    L = rng.integers(1500, 2049, size=60)
    _, sizes = _check(fr, L, 4096)
    assert sizes.max() <= 5120
    # ten 700-token sequences: the slab really follows the cap
    for cap in (1000, 2800):
        _, sizes = _check(fr, [700] * 10, cap)
        assert sizes.max() <= cap + cap // 4


@pytest.mark.parametrize("seed", range(20))
def test_random_length_mixes(fr, seed):
    rng = np.random.default_rng(seed)
    S = int(rng.integers(1, 400))
    L = rng.integers(0, int(rng.integers(1, 5000)), size=S)
    L[rng.uniform(size=S) < 0.1] = 0  # empty sequences
    for cap in (1, 256, 1000, 4096, 0):
        _check(fr, L, cap)


def test_empty_sequences_and_no_tokens(fr):
    begin, sizes = _check(fr, [0, 0, 50000, 0, 3, 0], 32768)
    assert np.all(sizes > 0)
    begin, sizes = _check(fr, [0, 0, 0], 0)  # T = 0: one slab without tokens
    assert begin == [0, 3] and list(sizes) == [0]
    a, _ = _args(fr, np.zeros(0, dtype=np.int64), 0)
    assert fr.slab_plan(a) == ([0], 0)


def test_default_slab_is_bounded_on_the_7b_workloads(fr):
    """The 7B workloads run as several slabs of at most 40960 tokens (E <= 12.5 GB)."""
    for c in (3, 4, 5):
        ro = make_rollouts(CONFIGS[c])
        # about half the trajectories are kept: their lengths have the same distribution
        L = ro.lengths[::2]
        begin, sizes = _check(fr, L, 0)
        assert len(sizes) >= 4 and sizes.max() <= 40960, (c, len(sizes), sizes.max())


def test_negative_slab_is_rejected(fr):
    a, _ = _args(fr, np.asarray([5, 6], dtype=np.int64), -1)
    assert fr._lib.fastrl_policy_loss_slab_plan(ctypes.byref(a), None, 0, None) == -3
