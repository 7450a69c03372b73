"""The gradient checks of the GPU parity tests (tests/_parity.py::check_grads), on the CPU.

The backward GEMMs read the one-hot term of dZ from the bf16 exp-logit operand, so the
softmax-part check allows the bound of that rounding (fold_bounds).  Here an emulation of
that arithmetic in float64 (bf16 exp-logits, the label entry E[t][y_t] - exp(lse_t) rounded
to bf16, dH = -c E' W, dW = -(c E')^T H with c_t = g_t exp(-lse_t)) must pass, and planted
mistakes in the softmax part of the oracle's own gradients must still fail: the part
dropped, its sign flipped, one vocabulary block of it 5% off, the one-hot term dropped."""
import numpy as np
import pytest
import torch

import oracle
from tests._parity import check_grads, fold_bounds, onehot_parts, BF16_U


def _bf16(x):
    return torch.from_numpy(np.asarray(x, dtype=np.float32)).bfloat16().double().numpy()


@pytest.fixture(scope="module", params=[(700, 64, 0.02), (1300, 136, 0.05)])
def case(request):
    V, d, w_std = request.param
    rng = np.random.default_rng(V + d)
    T = 300
    H = _bf16(rng.normal(size=(T, d)))
    W = _bf16(rng.normal(0.0, w_std, size=(V, d)))
    y = rng.integers(0, V, size=T)
    y[:40] = 3  # one label shared by many tokens
    x, lse = oracle.token_logprob(H, W, y)
    off = np.array([0, 50, 120, 200, 300])
    A = np.array([1.2, -0.7, 0.4, -1.5])
    old = x + rng.normal(0, 0.05, size=T)
    loss, g, _ = oracle.policy_loss(x, old, None, off, A, algo="grpo", norm="token_mean",
                                    eps_low=0.2, eps_high=0.2)
    dH, dW = oracle.lmhead_backward(H, W, y, lse, g)
    # the fold's arithmetic: bf16 exp-logits with the label entry folded in, fp64 GEMMs
    E = _bf16(np.exp(H @ W.T))
    E[np.arange(T), y] = _bf16(E[np.arange(T), y] - np.exp(lse))
    c = g * np.exp(-lse)
    dH_f = -c[:, None] * (E @ W)
    dW_f = -(c[:, None] * E).T @ H
    return dict(H=H, W=W, y=y, g=g, lse=lse, dH=dH, dW=dW, dH_f=dH_f, dW_f=dW_f)


def _check(k, dH, dW):
    return check_grads(k["H"], k["W"], k["y"], k["g"], dH, dW, k["dH"], k["dW"],
                       dg=np.zeros(len(k["y"])), lse=k["lse"])


def test_fold_emulation_passes_and_is_within_its_bound(case):
    errs = _check(case, case["dH_f"], case["dW_f"])
    bH, bW = fold_bounds(case["H"], case["W"], case["y"], case["g"], BF16_U)
    assert np.linalg.norm(case["dH_f"] - case["dH"]) <= bH + 1e-2 * np.linalg.norm(case["dH"])
    assert np.linalg.norm(case["dW_f"] - case["dW"]) <= bW + 1e-2 * np.linalg.norm(case["dW"])
    print(errs)


def _planted(k, which):
    dH1, dW1 = onehot_parts(k["H"], k["W"], k["y"], k["g"])
    sH, sW = k["dH"] - dH1, k["dW"] - dW1  # softmax parts
    if which == "drop_softmax":
        return dH1, dW1
    if which == "flip_softmax":
        return dH1 - sH, dW1 - sW
    if which == "block_5pct":  # dW's softmax part 5% too large in vocabulary rows 256..511
        dWm = k["dW"].copy()
        dWm[256:512] += 0.05 * sW[256:512]
        return k["dH"], dWm
    if which == "drop_onehot":
        return sH, sW
    raise ValueError(which)


@pytest.mark.parametrize("which", ["drop_softmax", "flip_softmax", "block_5pct", "drop_onehot"])
def test_planted_mistakes_fail(case, which):
    dH, dW = _planted(case, which)
    with pytest.raises(AssertionError):
        _check(case, dH, dW)
