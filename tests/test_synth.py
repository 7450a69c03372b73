"""The seeded rollout generator: determinism, shapes and distributions of the five
workloads, and the clip-edge margins it promises."""
import math

import numpy as np
import pytest

from synth import (CONFIGS, make_rollouts, make_dense, skew_tokens, TOKEN_EDGE_MARGIN,
                   SEQ_EDGE_MARGIN)


@pytest.mark.parametrize("c", [1, 2, 3])
def test_structure(c):
    cfg = CONFIGS[c]
    a = make_rollouts(cfg)
    b = make_rollouts(cfg)
    assert np.array_equal(a.token_ids, b.token_ids) and np.array_equal(a.rewards, b.rewards)
    assert a.N == sum(np.diff(a.group_off)) and len(a.lengths) == a.N
    assert a.lengths.min() >= cfg.len_lo and a.lengths.max() <= cfg.len_hi
    assert a.token_ids.min() >= 0 and a.token_ids.max() < cfg.V
    assert a.T_total == a.lengths.sum() == len(a.old_noise) == len(a.ref_noise)
    assert abs(a.old_noise.std() - 0.05) < 0.005
    lo, hi = math.log1p(-cfg.eps_low), math.log1p(cfg.eps_high)
    x = -a.old_noise
    assert np.all(np.abs(x - lo) >= TOKEN_EDGE_MARGIN) and np.all(np.abs(x - hi) >= TOKEN_EDGE_MARGIN)


def test_gspo_groups_and_seq_margin():
    cfg = CONFIGS[5]
    a = make_rollouts(cfg, Q=32)
    assert set(np.diff(a.group_off)) <= {8, 12, 16}
    lo, hi = math.log1p(-cfg.eps_low), math.log1p(cfg.eps_high)
    for i in range(a.N):
        m = -a.old_noise[a.traj_tok_off[i]:a.traj_tok_off[i + 1]].mean()
        assert abs(m - lo) >= SEQ_EDGE_MARGIN and abs(m - hi) >= SEQ_EDGE_MARGIN


def test_rewards_cfg3_values():
    a = make_rollouts(CONFIGS[3])
    assert set(np.unique(a.rewards)) <= {np.float32(0), np.float32(0.1), np.float32(1),
                                         np.float32(1.1)}


def test_dense_deterministic_small():
    torch = pytest.importorskip("torch")
    cfg = CONFIGS[1]
    H1, W1 = make_dense(cfg, 100, d=32, V=50)
    H2, W2 = make_dense(cfg, 100, d=32, V=50)
    assert torch.equal(H1, H2) and torch.equal(W1, W2)
    assert H1.dtype == torch.float32 and W1.shape == (50, 32)
    Hb, Wb = make_dense(CONFIGS[2], 10, d=16, V=8)
    assert Hb.dtype == torch.bfloat16


def test_skew_tokens_head_share():
    a = skew_tokens(make_rollouts(CONFIGS[3], Q=8), 0.7)
    b = skew_tokens(make_rollouts(CONFIGS[3], Q=8), 0.7)
    assert np.array_equal(a.token_ids, b.token_ids)
    share = float((a.token_ids == 0).mean())
    assert 0.68 < share < 0.72, share
    c = skew_tokens(make_rollouts(CONFIGS[3], Q=2), 1.0)
    assert (c.token_ids == 0).all()
