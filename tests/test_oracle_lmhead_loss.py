"""Pins for the oracle's LM-head log-probabilities, loss and backward: closed forms,
invariants, a library log_softmax, special cases that reduce one objective to
another, and central finite differences of the composite loss."""
import numpy as np
import pytest
import scipy.special

from oracle import token_logprob, lmhead_backward, policy_loss, token_weights, logits


def _rand(seed, T=12, d=16, V=64, scale=1.0):
    rng = np.random.default_rng(seed)
    H = rng.normal(size=(T, d))
    W = rng.normal(scale=0.3 * scale, size=(V, d))
    y = rng.integers(0, V, size=T)
    return H, W, y


def test_logprob_vs_scipy_and_normalisation():
    H, W, y = _rand(0, T=40, d=32, V=300)
    logp, lse = token_logprob(H, W, y, row_chunk=7)
    ref = scipy.special.log_softmax(H @ W.T, axis=1)
    np.testing.assert_allclose(logp, ref[np.arange(40), y], rtol=0, atol=1e-12)
    # every label at once: exp(logp) sums to one over the vocabulary
    allp = np.stack([token_logprob(H, W, np.full(40, v))[0] for v in range(300)], 1)
    np.testing.assert_allclose(np.exp(allp).sum(1), 1.0, atol=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(H @ W.T, axis=1), atol=1e-12)


def test_logprob_zero_weights_is_uniform():
    H, W, y = _rand(1, V=4096)
    logp, _ = token_logprob(H, np.zeros_like(W), y)
    assert np.all(logp == -np.log(4096.0))
    logp, _ = token_logprob(np.zeros_like(H), W, y)
    assert np.all(logp == -np.log(4096.0))


def test_logprob_large_logits_stable():
    H, W, y = _rand(2)
    logp, lse = token_logprob(H * 300.0, W, y)
    assert np.all(np.isfinite(logp)) and np.all(logp <= 0)


def _seq(seed, S=5, lmax=6):
    rng = np.random.default_rng(seed)
    L = rng.integers(1, lmax + 1, size=S)
    off = np.concatenate([[0], np.cumsum(L)])
    A = rng.normal(size=S)
    return off, A, rng


def test_loss_equals_minus_mean_adv_when_old_equals_new():
    off, A, rng = _seq(3, S=7)
    T = off[-1]
    x = rng.normal(-5, 1, size=T)
    L = np.diff(off)
    for algo in ("grpo", "dapo", "gspo"):
        loss, g, _ = policy_loss(x, x, None, off, A, algo=algo, norm="seq_mean_token_mean")
        assert abs(loss - (-A.mean())) < 1e-12
        loss, g, _ = policy_loss(x, x, None, off, A, algo=algo, norm="token_mean")
        assert abs(loss - (-(A * L).sum() / T)) < 1e-12


def test_kl_zero_when_ref_equals_new_and_positive_otherwise():
    off, A, rng = _seq(4)
    T = off[-1]
    x = rng.normal(-5, 1, size=T)
    o = x + rng.normal(0, 0.05, size=T)
    l0, g0, _ = policy_loss(x, o, None, off, A, beta=0.0)
    l1, g1, _ = policy_loss(x, o, x, off, A, beta=0.04)
    assert abs(l1 - l0) < 1e-14
    np.testing.assert_allclose(g1, g0, atol=1e-15)
    f = x + rng.normal(0, 0.3, size=T)
    l2, _, _ = policy_loss(x, o, f, off, A, beta=0.04)
    assert l2 > l0  # k3 >= 0


def test_dapo_symmetric_equals_grpo_token_mean():
    off, A, rng = _seq(5)
    T = off[-1]
    x = rng.normal(-5, 1, size=T)
    o = x + rng.normal(0, 0.3, size=T)
    a = policy_loss(x, o, None, off, A, algo="dapo", norm="token_mean", eps_low=0.2,
                    eps_high=0.2)
    b = policy_loss(x, o, None, off, A, algo="grpo", norm="token_mean", eps_low=0.2,
                    eps_high=0.2)
    assert a[0] == b[0]
    np.testing.assert_array_equal(a[1], b[1])


def test_gspo_single_token_equals_grpo_seq_mean():
    rng = np.random.default_rng(6)
    S = 9
    off = np.arange(S + 1)
    A = rng.normal(size=S)
    x = rng.normal(-5, 1, size=S)
    o = x + rng.normal(0, 0.3, size=S)
    a = policy_loss(x, o, None, off, A, algo="gspo", eps_low=0.2, eps_high=0.28)
    b = policy_loss(x, o, None, off, A, algo="grpo", eps_low=0.2, eps_high=0.28)
    assert abs(a[0] - b[0]) < 1e-14
    np.testing.assert_allclose(a[1], b[1], atol=1e-15)


def test_clip_indicator_inclusive_edge():
    # ratio exactly on an edge: c = 1 (Sec. 3.1 uses <= and >=), so the gradient flows
    x, o = np.asarray([0.1]), np.asarray([0.0])
    rho = float(np.exp(x - o)[0])
    e_hi = rho - 1.0  # exact (Sterbenz), so 1 + e_hi == rho
    assert 1.0 + e_hi == rho
    _, g, _ = policy_loss(x, o, None, [0, 1], [1.0], eps_low=0.2, eps_high=e_hi)
    assert g[0] == -rho
    _, g, _ = policy_loss(x + 1e-9, o, None, [0, 1], [1.0], eps_low=0.2, eps_high=e_hi)
    assert g[0] == 0.0
    x = np.asarray([-0.1])
    rho = float(np.exp(x - o)[0])
    e_lo = 1.0 - rho
    assert 1.0 - e_lo == rho
    _, g, _ = policy_loss(x, o, None, [0, 1], [-2.0], eps_low=e_lo, eps_high=0.2)
    assert g[0] == 2.0 * rho
    _, g, _ = policy_loss(x - 1e-9, o, None, [0, 1], [-2.0], eps_low=e_lo, eps_high=0.2)
    assert g[0] == 0.0


def test_token_weights():
    off = np.asarray([0, 2, 5, 5, 6])
    w = token_weights(off, "seq_mean_token_mean")
    np.testing.assert_allclose(w, [1 / 8, 1 / 8, 1 / 12, 1 / 12, 1 / 12, 1 / 4])
    w = token_weights(off, "token_mean")
    np.testing.assert_allclose(w, np.full(6, 1 / 6))


def test_lmhead_backward_invariants():
    H, W, y = _rand(8, T=20, d=12, V=50)
    _, lse = token_logprob(H, W, y)
    g = np.random.default_rng(8).normal(size=20)
    dH, dW = lmhead_backward(H, W, y, lse, g, row_chunk=6)
    # sum over the vocabulary of dZ is zero for every token
    np.testing.assert_allclose(dW.sum(0), 0.0, atol=1e-12 * np.abs(dW).max())
    # <dW, W> = <dH, H> = sum_t sum_v dZ_tv z_tv
    assert abs((dW * W).sum() - (dH * H).sum()) < 1e-10 * np.abs(dH * H).sum()
    # H = 0: dH_t = g_t (W_{y_t} - mean_v W_v)
    Z = np.zeros_like(H)
    _, lse0 = token_logprob(Z, W, y)
    dH0, _ = lmhead_backward(Z, W, y, lse0, g)
    np.testing.assert_allclose(dH0, g[:, None] * (W[y] - W.mean(0)), atol=1e-13)


def _composite(H, W, y, o, f, off, A, **kw):
    logp, _ = token_logprob(H, W, y)
    return policy_loss(logp, o, f, off, A, **kw)[0]


@pytest.mark.parametrize("algo,norm,beta,el,eh", [
    ("grpo", "seq_mean_token_mean", 0.04, 0.2, 0.2),
    ("grpo", "token_mean", 0.0, 0.2, 0.2),
    ("dapo", "token_mean", 0.0, 0.2, 0.28),
    ("gspo", "seq_mean_token_mean", 0.0, 3e-4, 4e-4),
    ("gspo", "token_mean", 0.02, 0.05, 0.05),
])
def test_finite_differences(algo, norm, beta, el, eh):
    rng = np.random.default_rng(11)
    S, d, V = 4, 16, 64
    L = rng.integers(2, 9, size=S)
    off = np.concatenate([[0], np.cumsum(L)])
    T = off[-1]
    H = rng.normal(size=(T, d))
    W = rng.normal(scale=0.3, size=(V, d))
    y = rng.integers(0, V, size=T)
    A = rng.normal(size=S)
    x, lse = token_logprob(H, W, y)
    # old log-probs: token ratios (or GSPO sequence ratios) well away from clip edges,
    # with a mix of clipped and unclipped terms
    if algo == "gspo":
        shift = np.repeat(rng.choice([-3 * eh, 0.0, 3 * el], size=S), L)
        o = x - shift
    else:
        o = x + rng.choice([-0.5, -0.05, 0.05, 0.5], size=T)
    f = x + rng.normal(0, 0.2, size=T)
    kw = dict(algo=algo, norm=norm, eps_low=el, eps_high=eh, beta=beta)
    loss, g, _ = policy_loss(x, o, f, off, A, **kw)
    dH, dW = lmhead_backward(H, W, y, lse, g)
    h = 1e-6
    # dL/dlogp
    for t in range(T):
        xp, xm = x.copy(), x.copy()
        xp[t] += h
        xm[t] -= h
        fd = (policy_loss(xp, o, f, off, A, **kw)[0] - policy_loss(xm, o, f, off, A, **kw)[0]) / (2 * h)
        assert abs(fd - g[t]) < 1e-6 * max(1.0, abs(g[t])), (t, fd, g[t])
    # dL/dH and dL/dW on a sample of coordinates
    for _ in range(25):
        t, k = rng.integers(0, T), rng.integers(0, d)
        Hp, Hm = H.copy(), H.copy()
        Hp[t, k] += h
        Hm[t, k] -= h
        fd = (_composite(Hp, W, y, o, f, off, A, **kw) - _composite(Hm, W, y, o, f, off, A, **kw)) / (2 * h)
        assert abs(fd - dH[t, k]) < 1e-6 * max(1e-3, abs(dH[t, k])) + 1e-9, (t, k, fd, dH[t, k])
        v, k = rng.integers(0, V), rng.integers(0, d)
        Wp, Wm = W.copy(), W.copy()
        Wp[v, k] += h
        Wm[v, k] -= h
        fd = (_composite(H, Wp, y, o, f, off, A, **kw) - _composite(H, Wm, y, o, f, off, A, **kw)) / (2 * h)
        assert abs(fd - dW[v, k]) < 1e-6 * max(1e-3, abs(dW[v, k])) + 1e-9, (v, k, fd, dW[v, k])


def test_autograd_crosscheck():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(12)
    S, d, V = 3, 8, 32
    L = np.asarray([3, 1, 5])
    off = np.concatenate([[0], np.cumsum(L)])
    T = off[-1]
    H = rng.normal(size=(T, d))
    W = rng.normal(scale=0.3, size=(V, d))
    y = rng.integers(0, V, size=T)
    A = rng.normal(size=S)
    x, lse = token_logprob(H, W, y)
    o = x + rng.choice([-0.5, 0.05, 0.5], size=T)
    f = x + 0.1
    loss, g, _ = policy_loss(x, o, f, off, A, beta=0.04)
    dH, dW = lmhead_backward(H, W, y, lse, g)
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    lp = torch.log_softmax(Ht @ Wt.T, dim=1)[torch.arange(T), torch.tensor(y)]
    w = torch.tensor(token_weights(off, "seq_mean_token_mean"))
    At = torch.tensor(np.repeat(A, L))
    rho = torch.exp(lp - torch.tensor(o))
    sur = torch.minimum(rho * At, torch.clamp(rho, 0.8, 1.2) * At)
    ft = torch.tensor(f)
    k3 = torch.exp(ft - lp) - (ft - lp) - 1
    tl = (w * (-sur + 0.04 * k3)).sum()
    tl.backward()
    assert abs(tl.item() - loss) < 1e-12
    np.testing.assert_allclose(Ht.grad.numpy(), dH, atol=1e-12)
    np.testing.assert_allclose(Wt.grad.numpy(), dW, atol=1e-12)


def test_dW_rows_match_full_backward_and_finite_differences():
    """lmhead_dW_rows (exact dW rows for chosen vocabulary ids, used where the full dW is
    too large to form) equals the rows of the full backward, for ids that are labels, ids
    that are not, repeated ids and any chunking; and its rows are the central finite
    differences of the composite loss w.r.t. those rows of W."""
    from oracle.lmhead import lmhead_dW_rows
    rng = np.random.default_rng(13)
    S, d, V = 5, 12, 40
    L = rng.integers(2, 7, size=S)
    off = np.concatenate([[0], np.cumsum(L)])
    T = off[-1]
    H = rng.normal(size=(T, d))
    W = rng.normal(scale=0.3, size=(V, d))
    y = rng.integers(0, V // 2, size=T)  # the upper half of the vocabulary is never a label
    A = rng.normal(size=S)
    x, lse = token_logprob(H, W, y)
    o = x + rng.choice([-0.5, -0.05, 0.05, 0.5], size=T)
    f = x + rng.normal(0, 0.2, size=T)
    kw = dict(algo="grpo", norm="seq_mean_token_mean", eps_low=0.2, eps_high=0.2, beta=0.04)
    _, g, _ = policy_loss(x, o, f, off, A, **kw)
    _, dW = lmhead_backward(H, W, y, lse, g)
    rows = np.asarray([int(y[0]), int(y[3]), V - 1, V // 2 + 1, int(y[0]), 0])
    for chunk in (1, 3, T, 4096):
        got = lmhead_dW_rows(H, W, y, lse, g, rows, row_chunk=chunk)
        np.testing.assert_allclose(got, dW[rows], rtol=0, atol=1e-14)
    got = lmhead_dW_rows(H, W, y, lse, g, rows)
    h = 1e-6
    for r, v in enumerate(rows[:4]):
        for k in rng.choice(d, size=3, replace=False):
            Wp, Wm = W.copy(), W.copy()
            Wp[v, k] += h
            Wm[v, k] -= h
            fd = (_composite(H, Wp, y, o, f, off, A, **kw) -
                  _composite(H, Wm, y, o, f, off, A, **kw)) / (2 * h)
            assert abs(fd - got[r, k]) < 1e-6 * max(1e-3, abs(got[r, k])) + 1e-9, (v, k)
