"""GPU parity of the continuous-reward advantage groups (|A_i - A_j| < eps, appendix on the
grounding task) and of Alg. 1's |A|-descending traversal, through fastrl_prune_ex, against
the oracle on the same seeded inputs.  Bars: advantages bit-exact (float32), class ids, masks,
counts and compaction outputs bit-exact."""
import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, make_rollouts, make_dense, continuous_rewards, plant_duplicates
from tests._parity import to_dev, LOGP_ATOL, REL, check_grads, rel_fro

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


def _status():
    return torch.zeros(1, dtype=torch.int32, device=DEV)


def _continuous_batch(c, Q=None, seed=0, len_range=None, V=None, dup=True):
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg, Q=Q, len_range=len_range, V=V)
    if dup:
        plant_duplicates(ro, p_copy=0.7, p_mutate=0.2, seed=seed)
    ro.rewards = continuous_rewards(ro.group_off, seed=100 + seed)
    return cfg, ro


@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("kind", ["discrete", "continuous"])
def test_advantage_bit_exact(fr, c, kind):
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg)
    if kind == "continuous":
        ro.rewards = continuous_rewards(ro.group_off, seed=c)
    adv, cls, valid = oracle.group_advantage(ro.rewards, ro.group_off,
                                             drop_uniform=cfg.drop_uniform)
    st = _status()
    a, k, v = fr.advantage(to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV),
                           drop_uniform=cfg.drop_uniform, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    assert np.array_equal(a.cpu().numpy(), adv.astype(np.float32))
    assert np.array_equal(k.cpu().numpy(), cls)
    assert np.array_equal(v.cpu().numpy(), valid)


def _prune_ex(fr, ro, adv, cls, valid, V, *, eps, keep, n=1, tau=(4, 5)):
    st = _status()
    out = fr.prune(to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV),
                   to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV),
                   None if cls is None else to_dev(cls, DEV), to_dev(valid, DEV), V=V,
                   max_group=int(np.diff(ro.group_off).max()), max_len=int(ro.lengths.max()),
                   ngram_n=n, tau=tau, keep_ratio=keep, adv=to_dev(adv, DEV), group_eps=eps,
                   class_out=True, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    return out


def _check(out, ref, classes):
    N = len(ref["keep_mask"])
    assert np.array_equal(out["class_id"][:N].cpu().numpy(), classes)
    assert np.array_equal(out["keep_mask"].cpu().numpy(), ref["keep_mask"])
    assert np.array_equal(out["mdap_count"].cpu().numpy(), ref["mdap_count"])
    nk, tk = out["counts"].cpu().tolist()
    assert nk == len(ref["kept_traj"]) and tk == len(ref["tok_src"])
    assert np.array_equal(out["kept_traj"][:nk].cpu().numpy(), ref["kept_traj"])
    assert np.array_equal(out["kept_tok_off"][:nk + 1].cpu().numpy(), ref["kept_tok_off"])
    assert np.array_equal(out["tok_src"][:tk].cpu().numpy(), ref["tok_src"])


@pytest.mark.parametrize("eps", [1e-4, 1e-3, 3e-2])
@pytest.mark.parametrize("keep", [0.0, 0.4])
@pytest.mark.parametrize("tau", [(4, 5), (2, 1)])
def test_prune_continuous_groups(fr, eps, keep, tau):
    cfg, ro = _continuous_batch(5, Q=40, seed=int(eps * 1e5), len_range=(1, 48), V=64)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=keep, group_eps=eps,
                               tau_num=tau[0], tau_den=tau[1])
    adv32 = ref["adv"].astype(np.float32)
    out = _prune_ex(fr, ro, adv32, None, ref["group_valid"], 64, eps=eps, keep=keep, tau=tau)
    _check(out, ref, ref["prune_class"])
    # the groups really merge distinct rewards at this eps, and prune something
    merged = sum(len(set(ref["prune_class"][a:b])) < len(set(ro.rewards[a:b]))
                 for a, b in zip(ro.group_off[:-1], ro.group_off[1:]))
    assert merged > 0
    if keep == 0.0 and tau == (4, 5):
        assert ref["keep_mask"].sum() < ro.N


@pytest.mark.parametrize("c", [2, 3, 4, 5])
def test_prune_continuous_full_size(fr, c):
    """Continuous rewards on each workload's full batch structure (eps = 1e-4)."""
    cfg, ro = _continuous_batch(c, seed=c, dup=False)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=cfg.keep_ratio, group_eps=1e-4,
                               drop_uniform=cfg.drop_uniform)
    out = _prune_ex(fr, ro, ref["adv"].astype(np.float32), None, ref["group_valid"], cfg.V,
                    eps=1e-4, keep=cfg.keep_ratio)
    _check(out, ref, ref["prune_class"])


@pytest.mark.parametrize("c", [3, 5])
def test_discrete_classes_with_advantage_order_unchanged(fr, c):
    """Bit-equal classes traversed by |A| descending == ascending index (fastrl_prune)."""
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg, Q=32, len_range=(1, 40), V=40)
    plant_duplicates(ro, p_copy=0.7, p_mutate=0.2, seed=c)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=cfg.keep_ratio,
                               drop_uniform=cfg.drop_uniform)
    adv32 = ref["adv"].astype(np.float32)
    out = _prune_ex(fr, ro, adv32, ref["class_id"], ref["group_valid"], 40, eps=0.0,
                    keep=cfg.keep_ratio)
    _check(out, ref, ref["class_id"])
    plain = fr.prune(to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV),
                     to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV),
                     to_dev(ref["class_id"], DEV), to_dev(ref["group_valid"], DEV), V=40,
                     max_group=int(np.diff(ro.group_off).max()), max_len=40,
                     keep_ratio=cfg.keep_ratio)
    torch.cuda.synchronize()
    assert np.array_equal(plain["keep_mask"].cpu().numpy(), out["keep_mask"].cpu().numpy())


def test_nonfinite_advantage_flags_and_stays_valid(fr):
    cfg, ro = _continuous_batch(1, seed=3, dup=False)
    adv = oracle.group_advantage(ro.rewards, ro.group_off)[0].astype(np.float32)
    adv[3] = np.nan
    adv[9] = np.inf
    st = _status()
    out = fr.prune(to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV),
                   to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV), None, None, V=cfg.V,
                   max_group=8, max_len=64, keep_ratio=0.5, adv=to_dev(adv, DEV),
                   group_eps=1e-4, class_out=True, status=st)
    torch.cuda.synchronize()
    assert st.item() & 0x10  # FASTRL_SB_BAD_REWARD
    cls = out["class_id"][:ro.N].cpu().numpy()
    for a, b in zip(ro.group_off[:-1], ro.group_off[1:]):
        assert cls[a:b].min() == 0 and cls[a:b].max() < b - a
    # the budget still keeps K_q per question
    keep = out["keep_mask"].cpu().numpy()
    for a, b in zip(ro.group_off[:-1], ro.group_off[1:]):
        assert keep[a:b].sum() == 4


def test_hot_path_step_continuous_small(fr):
    """End to end under continuous groups: pruning bit-exact, log-probs, loss, dH, dW."""
    cfg = CONFIGS[1]
    ro = make_rollouts(cfg)
    plant_duplicates(ro, p_copy=0.5, p_mutate=0.3, seed=11)
    ro.rewards = continuous_rewards(ro.group_off, seed=11)
    pr = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                              lmhead=False, keep_ratio=cfg.keep_ratio, group_eps=1e-4)
    src = pr["tok_src"]
    H, W = make_dense(cfg, ro.T_total, device="cpu")
    H64, W64 = H.double().numpy(), W.double().numpy()
    y = ro.token_ids[src].astype(np.int64)
    lp, lse = oracle.token_logprob(H64[src], W64, y)
    old = np.full(ro.T_total, np.nan)
    old[src] = lp + ro.old_noise[src]
    old = old.astype(np.float32)
    loss, g, _ = oracle.policy_loss(lp, old[src].astype(np.float64), None, pr["kept_tok_off"],
                                    pr["adv"][pr["kept_traj"]], algo=cfg.algo, norm=cfg.norm,
                                    eps_low=cfg.eps_low, eps_high=cfg.eps_high, beta=0.0)
    dH, dW = oracle.lmhead_backward(H64[src], W64, y, lse, g)
    st = _status()
    out = fr.hot_path_step(to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV),
                           to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV),
                           H.to(DEV), W.to(DEV), to_dev(old, DEV), V=cfg.V, max_group=8,
                           max_len=int(ro.lengths.max()), keep_ratio=cfg.keep_ratio,
                           group_eps=1e-4, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    assert np.array_equal(out["prune"]["keep_mask"].cpu().numpy(), pr["keep_mask"])
    T = out["t_kept"]
    assert T == len(src)
    call = out["call"]
    assert np.abs(call.logp[:T].double().cpu().numpy() - lp).max() < LOGP_ATOL
    assert abs(float(call.loss.item()) - loss) <= REL * max(abs(loss), 1e-8)
    assert rel_fro(call.dhidden[:T].double().cpu().numpy(), dH) < REL
    assert rel_fro(call.dW.double().cpu().numpy(), dW) < REL
