"""Property-based GPU parity (hypothesis, derandomized so every run draws the same cases):
random small batches with ragged groups (1 to 24 rollouts), trajectories shorter than the
n-gram length (0 to 12 tokens), all-equal reward groups, zero-advantage classes, tiny
vocabularies (many repeated n-grams, so MDAP prunes) and every tau, through pruning
(bit-exact against the oracle) and, on the kept tokens, through the loss forward/backward with
one-token and empty sequences (log-probs, loss, clip count, gradients against the oracle)."""
import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st, HealthCheck

import oracle
from synth import CONFIGS, Rollouts
from tests._parity import to_dev, check_grads, g_deviation, LOGP_ATOL, REL

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SETTINGS = settings(max_examples=40, derandomize=True, deadline=None,
                    suppress_health_check=list(HealthCheck))


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


@st.composite
def batches(draw):
    Q = draw(st.integers(1, 6))
    G = draw(st.lists(st.integers(1, 24), min_size=Q, max_size=Q))
    N = sum(G)
    lengths = draw(st.lists(st.integers(0, 12), min_size=N, max_size=N))
    V = draw(st.sampled_from([3, 7, 50]))
    reward_set = draw(st.sampled_from([(0.0,), (0.0, 1.0), (0.0, 0.5, 1.0), (0.25, 1.1, 2.0, 3.5)]))
    seed = draw(st.integers(0, 2**31 - 1))
    rng = np.random.default_rng(seed)
    group_off = np.concatenate([[0], np.cumsum(G)]).astype(np.int32)
    traj_tok_off = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int64)
    rewards = rng.choice(np.asarray(reward_set, dtype=np.float32), size=N)
    # some questions with all-equal rewards (advantage 0 for every member)
    for q in range(Q):
        if rng.uniform() < 0.3:
            rewards[group_off[q]:group_off[q + 1]] = rewards[group_off[q]]
    T = int(traj_tok_off[-1])
    tokens = rng.integers(0, V, size=T).astype(np.int32)
    n = draw(st.integers(1, 3))
    tau = draw(st.sampled_from([(0, 1), (1, 2), (4, 5), (1, 1), (2, 1)]))
    keep = draw(st.sampled_from([0.0, 0.5]))
    ro = Rollouts(CONFIGS[3], group_off, traj_tok_off, np.asarray(lengths, dtype=np.int64),
                  rewards, tokens, rng.normal(0, 0.05, size=T), rng.normal(0, 0.05, size=T),
                  extra={"V": V, "seed": seed})
    return ro, V, n, tau, keep


@SETTINGS
@given(batches())
def test_prune_properties(fr, case):
    ro, V, n, tau, keep = case
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, ngram_n=n, tau_num=tau[0], tau_den=tau[1],
                               keep_ratio=keep)
    stw = torch.zeros(1, dtype=torch.int32, device=DEV)
    adv, cls, valid = fr.advantage(to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV), status=stw)
    out = fr.prune(to_dev(ro.token_ids, DEV) if ro.T_total else torch.zeros(1, dtype=torch.int32, device=DEV),
                   to_dev(ro.traj_tok_off, DEV), to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV),
                   cls, valid, V=V, max_group=int(np.diff(ro.group_off).max()),
                   max_len=max(int(ro.lengths.max()), 1), ngram_n=n, tau=tau, keep_ratio=keep,
                   status=stw)
    torch.cuda.synchronize()
    assert stw.item() == 0, fr.status_names(stw.item())
    assert np.array_equal(cls.cpu().numpy(), ref["class_id"])
    assert np.array_equal(out["keep_mask"].cpu().numpy(), ref["keep_mask"])
    assert np.array_equal(out["mdap_count"].cpu().numpy(), ref["mdap_count"])
    nk, tk = out["counts"].cpu().tolist()
    assert (nk, tk) == (len(ref["kept_traj"]), len(ref["tok_src"]))
    assert np.array_equal(out["kept_traj"][:nk].cpu().numpy(), ref["kept_traj"])
    assert np.array_equal(out["kept_tok_off"][:nk + 1].cpu().numpy(), ref["kept_tok_off"])
    assert np.array_equal(out["tok_src"][:tk].cpu().numpy(), ref["tok_src"])


@st.composite
def loss_cases(draw):
    S = draw(st.integers(1, 12))
    L = draw(st.lists(st.integers(0, 40), min_size=S, max_size=S))
    algo = draw(st.sampled_from(["grpo", "dapo", "gspo"]))
    norm = draw(st.sampled_from(["seq_mean_token_mean", "token_mean"]))
    beta = draw(st.sampled_from([0.0, 0.04]))
    V = draw(st.sampled_from([257, 700, 1300]))
    d = draw(st.sampled_from([64, 136]))
    slab = draw(st.sampled_from([0, 16, 100]))
    seed = draw(st.integers(0, 2**31 - 1))
    return S, np.asarray(L), algo, norm, beta, V, d, slab, seed


@SETTINGS
@given(loss_cases())
def test_loss_properties(fr, case):
    S, L, algo, norm, beta, V, d, slab, seed = case
    rng = np.random.default_rng(seed)
    off = np.concatenate([[0], np.cumsum(L)]).astype(np.int64)
    T = int(off[-1])
    eps = {"grpo": (0.2, 0.2), "dapo": (0.2, 0.28), "gspo": (3e-4, 4e-4)}[algo]
    H = torch.from_numpy(rng.normal(size=(max(T, 1), d)).astype(np.float32)).bfloat16()
    W = torch.from_numpy(rng.normal(0, 0.05, size=(V, d)).astype(np.float32)).bfloat16()
    y = rng.integers(0, V, size=max(T, 1)).astype(np.int32)
    A = rng.choice([-1.5, -0.3, 0.0, 0.7, 2.0], size=S).astype(np.float32)
    H64, W64 = H.double().numpy(), W.double().numpy()
    x, lse = oracle.token_logprob(H64[:T], W64, y[:T])
    # old log-probs: token ratios (GSPO: sequence ratios) kept >= 1e-3 away from the clip edges
    if algo == "gspo":
        shift = rng.choice([-2e-3, 0.0, 1e-4, -1e-4, 3e-3], size=S)
        o = x - np.repeat(shift, L)
    else:
        o = x - rng.choice([-0.5, -0.1, 0.0, 0.05, 0.3], size=T)
    f = x + rng.normal(0, 0.05, size=T)
    kw = dict(algo=algo, norm=norm, eps_low=eps[0], eps_high=eps[1], beta=beta)
    loss, g, info = oracle.policy_loss(x, o, f if beta else None, off, A, **kw)
    dH, dW = oracle.lmhead_backward(H64[:T], W64, y[:T], lse, g)
    stw = torch.zeros(1, dtype=torch.int32, device=DEV)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    call = fr.LossCall(H.to(DEV), W.to(DEV), t(y), t(np.concatenate([o, [0.0]]).astype(np.float32)),
                       t(off), torch.from_numpy(off), t(A),
                       ref_logp=t(np.concatenate([f, [0.0]]).astype(np.float32)) if beta else None,
                       status=stw, slab_tokens=slab, T=T, **kw).run()
    torch.cuda.synchronize()
    assert stw.item() == 0, fr.status_names(stw.item())
    assert abs(call.loss.item() - loss) <= REL * max(abs(loss), 1e-6) + 1e-7, (call.loss.item(), loss)
    assert int(call.stats[0].item()) == info["clipped_tokens"]
    if T == 0:
        assert torch.count_nonzero(call.dW).item() == 0
        return
    assert np.abs(call.logp[:T].double().cpu().numpy() - x).max() < LOGP_ATOL
    dg = g_deviation(x, o, f if beta else None, off, A, **kw)
    check_grads(H64[:T], W64, y[:T], g, call.dhidden[:T].double().cpu().numpy(),
                call.dW.double().cpu().numpy(), dH, dW, dg=dg, lse=lse)


@st.composite
def logprob_cases(draw):
    rows = draw(st.integers(1, 300))
    T = draw(st.integers(0, 400))
    V = draw(st.sampled_from([1, 2, 7, 255, 256, 257, 1000, 2600]))
    d = draw(st.sampled_from([8, 64, 136, 264]))
    dtype = draw(st.sampled_from(["bf16", "f32"]))
    gather = draw(st.booleans())
    scale = draw(st.sampled_from([1.0, 30.0]))
    seed = draw(st.integers(0, 2**31 - 1))
    return rows, T, V, d, dtype, gather, scale, seed


@SETTINGS
@given(logprob_cases())
def test_token_logprob_properties(fr, case):
    """fastrl_token_logprob and fastrl_token_logprob_noalloc on random shapes: vocabularies
    from 1 to 2600 (ragged last vocabulary block), hidden sizes 8 to 264, gathered rows with
    repeats or the first T rows, both dtypes, logits of magnitude ~1 or ~100; log-probs and
    log-sum-exps against the oracle, the two entry points identical."""
    rows, T, V, d, dtype, gather, scale, seed = case
    if not gather:
        T = min(T, rows)
    rng = np.random.default_rng(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    H = torch.from_numpy(rng.normal(0, scale, size=(rows, d)).astype(np.float32)).to(tdt)
    W = torch.from_numpy(rng.normal(0, 0.05, size=(V, d)).astype(np.float32)).to(tdt)
    y = rng.integers(0, V, size=rows).astype(np.int32)
    idx = rng.integers(0, rows, size=T).astype(np.int32) if gather else np.arange(T, dtype=np.int32)
    H64, W64 = H.double().numpy(), W.double().numpy()
    lp_ref, lse_ref = oracle.token_logprob(H64[idx], W64, y[idx].astype(np.int64))
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    st_ = torch.zeros(1, dtype=torch.int32, device=DEV)
    ri = t(idx) if gather else None
    lp, lse = fr.token_logprob(H.to(DEV), W.to(DEV), t(y), row_index=ri, T=T, status=st_)
    lp2 = torch.full((max(T, 1),), float("nan"), device=DEV)
    lse2 = torch.full((max(T, 1),), float("nan"), device=DEV)
    fr.token_logprob_noalloc(H.to(DEV), W.to(DEV), t(y), lp2, lse2, row_index=ri, T=T,
                             status=st_)
    torch.cuda.synchronize()
    assert st_.item() == 0, fr.status_names(st_.item())
    if T == 0:
        return
    assert np.abs(lp.double().cpu().numpy() - lp_ref).max() < LOGP_ATOL
    assert np.abs(lse.double().cpu().numpy() - lse_ref).max() < LOGP_ATOL
    assert torch.equal(lp, lp2[:T]) and torch.equal(lse, lse2[:T])
