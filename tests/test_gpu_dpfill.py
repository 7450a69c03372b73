"""GPU parity of Alg. 1's DP-alignment fill (fastrl_prune_ex with dp_align = d) against the
oracle: keep mask, compaction outputs bit-exact; the kept count a multiple of d."""
import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, make_rollouts, continuous_rewards
from tests._parity import to_dev

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


def _run(fr, ro, cfg, d, *, group_eps=0.0, keep=None):
    keep = cfg.keep_ratio if keep is None else keep
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=keep, drop_uniform=cfg.drop_uniform,
                               group_eps=group_eps, dp_align=d)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    t = lambda x: to_dev(x, DEV)
    out = fr.prune(t(ro.token_ids), t(ro.traj_tok_off), t(ro.rewards), t(ro.group_off),
                   t(ref["class_id"]), t(ref["group_valid"]), V=int(ro.extra["V"]),
                   max_group=int(np.diff(ro.group_off).max()), max_len=int(ro.lengths.max()),
                   keep_ratio=keep, adv=t(ref["adv"].astype(np.float32)), group_eps=group_eps,
                   dp_align=d, status=st)
    torch.cuda.synchronize()
    return ref, out, st.item()


def _check(ref, out):
    assert np.array_equal(out["keep_mask"].cpu().numpy(), ref["keep_mask"])
    assert np.array_equal(out["mdap_count"].cpu().numpy(), ref["mdap_count"])
    nk, tk = out["counts"].cpu().tolist()
    assert nk == len(ref["kept_traj"]) and tk == len(ref["tok_src"])
    assert np.array_equal(out["kept_traj"][:nk].cpu().numpy(), ref["kept_traj"])
    assert np.array_equal(out["kept_tok_off"][:nk + 1].cpu().numpy(), ref["kept_tok_off"])
    assert np.array_equal(out["tok_src"][:tk].cpu().numpy(), ref["tok_src"])


@pytest.mark.parametrize("c", [2, 3, 4, 5])
@pytest.mark.parametrize("d", [2, 3, 8, 96])
def test_dp_fill_full_size(fr, c, d):
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg)
    ref, out, st = _run(fr, ro, cfg, d, keep=0.37 if c != 5 else None)
    assert st == 0
    _check(ref, out)
    assert int(ref["keep_mask"].sum()) % d == 0


def test_dp_fill_with_continuous_groups_and_pure_mdap(fr):
    cfg = CONFIGS[3]
    ro = make_rollouts(cfg, Q=24, len_range=(4, 40), V=50)
    ro.rewards = continuous_rewards(ro.group_off, seed=4)
    for d in (5, 7):
        ref, out, st = _run(fr, ro, cfg, d, group_eps=1e-4, keep=0.0)
        assert st == 0
        _check(ref, out)
        assert ref["dp_added"] > 0 or int(ref["keep_mask"].sum()) % d == 0


def test_dp_fill_short_sets_status(fr):
    cfg = CONFIGS[1]
    ro = make_rollouts(cfg)  # 32 trajectories
    ref, out, st = _run(fr, ro, cfg, 4096, keep=0.5)
    assert st & 0x100
    _check(ref, out)
    assert int(out["counts"][0].item()) == int(ref["group_valid"].astype(bool).sum()) * 8
