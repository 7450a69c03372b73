"""Hand-derived fixtures for the two parts of the loss that the objective reductions do not
reach: the GSPO sequence ratio on sequences longer than one token (exp of the MEAN token
log-ratio, which one-token sequences cannot tell from the sum or from the mean of the token
ratios), and the direction of the KL estimator, fixed by the gradient of Sec. 3.1.

The checks take the loss function as an argument, so ``test_oracle_mutations`` can run them
against copies of the oracle with a planted mistake and see them fail."""
import json
import os

import numpy as np

from oracle import policy_loss

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def gspo_inputs(fx):
    o0 = fx["old_logp"]
    deltas = [np.asarray(s["delta"], dtype=np.float64) for s in fx["sequences"]]
    L = [len(d) for d in deltas]
    off = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
    o = np.full(off[-1], o0)
    x = o + np.concatenate(deltas)
    A = np.asarray([s["adv"] for s in fx["sequences"]], dtype=np.float64)
    return x, o, off, A


def check_gspo_golden(loss_fn):
    fx = _load("gspo_sequence.json")
    x, o, off, A = gspo_inputs(fx)
    for norm, exp in fx["expected"].items():
        loss, g, info = loss_fn(x, o, None, off, A, algo="gspo", norm=norm,
                                eps_low=fx["eps_low"], eps_high=fx["eps_high"], beta=0.0)
        assert abs(loss - exp["loss"]) <= 1e-12, (norm, loss, exp["loss"])
        np.testing.assert_allclose(g, exp["g"], rtol=0, atol=1e-12, err_msg=norm)
        assert info["clipped_tokens"] == exp["clipped_tokens"], (norm, info["clipped_tokens"])
    # sequence ratios exactly on a clip edge (Sec. 3.1: inclusive indicator, so the
    # gradient still flows): four log-ratios of +-1/8 have an exact mean, and the edge is
    # set to that s (s - 1 and 1 - s are exact by Sterbenz)
    off = np.asarray([0, 4], dtype=np.int64)
    o = np.full(4, -2.0)
    for sign, A in ((1.0, 1.0), (-1.0, -1.0)):
        x = o + sign * 0.125
        s = float(np.exp(sign * 0.125))
        el, eh = (0.2, s - 1.0) if sign > 0 else (1.0 - s, 0.2)
        _, g, info = loss_fn(x, o, None, off, [A], algo="gspo", norm="seq_mean_token_mean",
                             eps_low=el, eps_high=eh, beta=0.0)
        np.testing.assert_allclose(g, np.full(4, -s * A / 4), rtol=0, atol=1e-15)
        assert info["clipped_tokens"] == 0
        # one step past the edge: clipped, no gradient
        _, g, info = loss_fn(x + sign * 1e-9, o, None, off, [A], algo="gspo",
                             norm="seq_mean_token_mean", eps_low=el, eps_high=eh, beta=0.0)
        assert np.all(g == 0.0) and info["clipped_tokens"] == 4


def kl_inputs(fx):
    x = np.asarray(fx["logp"], dtype=np.float64)
    f = x + np.log(np.asarray(fx["ratio_ref_over_theta"], dtype=np.float64))
    off = np.asarray([0, len(x)], dtype=np.int64)
    return x, f, off


def check_kl_golden(loss_fn):
    fx = _load("kl_k3.json")
    x, f, off = kl_inputs(fx)
    beta = fx["beta"]
    exp = fx["expected"]
    # A = 0: the surrogate term vanishes, loss and g are the KL part alone
    loss, g, _ = loss_fn(x, x, f, off, [0.0], algo="grpo", norm="seq_mean_token_mean",
                         eps_low=0.2, eps_high=0.2, beta=beta)
    assert abs(loss - exp["loss"]) <= 1e-14, (loss, exp["loss"])
    np.testing.assert_allclose(g, exp["g"], rtol=0, atol=1e-15)
    # A != 0, unclipped ratios (old = x - 0.05): the KL part of g is g(beta) - g(0), and
    # equals -beta w_t (pi_ref/pi_theta - 1) whatever the surrogate does
    o = x - 0.05
    _, g1, _ = loss_fn(x, o, f, off, [0.8], algo="grpo", norm="seq_mean_token_mean",
                       eps_low=0.2, eps_high=0.2, beta=beta)
    _, g0, _ = loss_fn(x, o, None, off, [0.8], algo="grpo", norm="seq_mean_token_mean",
                       eps_low=0.2, eps_high=0.2, beta=0.0)
    w = 1.0 / len(x)
    ratio = np.asarray(fx["ratio_ref_over_theta"])
    np.testing.assert_allclose(g1 - g0, -beta * w * (ratio - 1.0), rtol=0, atol=1e-15)
    # the GSPO path adds the same token-level KL part
    _, g2, _ = loss_fn(x, o, f, off, [0.8], algo="gspo", norm="seq_mean_token_mean",
                       eps_low=0.2, eps_high=0.2, beta=beta)
    _, g3, _ = loss_fn(x, o, None, off, [0.8], algo="gspo", norm="seq_mean_token_mean",
                       eps_low=0.2, eps_high=0.2, beta=0.0)
    np.testing.assert_allclose(g2 - g3, -beta * w * (ratio - 1.0), rtol=0, atol=1e-15)


def test_gspo_sequence_ratio_golden():
    check_gspo_golden(policy_loss)


def test_kl_direction_golden():
    check_kl_golden(policy_loss)


def test_gspo_fixture_is_consistent():
    """The fixture's own arithmetic: each s is e to the mean delta, on the stated side of
    its clip edge, and the sum-of-log-ratios form would land on the other side."""
    fx = _load("gspo_sequence.json")
    lo, hi = 1.0 - fx["eps_low"], 1.0 + fx["eps_high"]
    for s in fx["sequences"]:
        d = np.asarray(s["delta"])
        assert abs(np.exp(d.mean()) - s["s"]) < 1e-15
        inside = (s["adv"] >= 0 and s["s"] <= hi) or (s["adv"] < 0 and s["s"] >= lo)
        assert inside == bool(s["c"])
    d0, d1 = (np.asarray(fx["sequences"][i]["delta"]) for i in (0, 1))
    assert np.exp(d0.sum()) > hi and np.exp(d1.sum()) < lo
    d3 = np.asarray(fx["sequences"][3]["delta"])
    assert np.exp(d3).mean() > hi
