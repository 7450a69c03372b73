"""GPU parity of the per-token policy entropy fused into the log-sum-exp pass of
fastrl_policy_loss_fwd_bwd (H_t = lse_t - sum_v p_v z_v from one extra partial sum per
vocabulary block) against the oracle's -sum p log p.  Bars: 2e-3 absolute per token (the
log-prob bar; entropies are O(log V)), 1e-4 relative on the fixed-order sum."""
import numpy as np
import pytest
import torch

import oracle
from tests._parity import Problem, to_dev, LOGP_ATOL

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ENT_ATOL = 2e-3

CASES = {
    "grpo_kl_bf16": (3, dict(Q=6, len_range=(20, 90), V=1000, d=136)),
    "gspo_bf16": (5, dict(Q=6, len_range=(30, 100), V=900, d=96)),
    "grpo_f32": (1, dict(Q=4, len_range=(16, 64), V=1500, d=72)),
}


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


def _call(fr, pb, *, backward, slab=0, status=None):
    cfg = pb.cfg
    pr = pb.pr
    return fr.LossCall(
        pb.H_poisoned.to(DEV), pb.W.to(DEV), to_dev(pb.ro.token_ids, DEV), to_dev(pb.old, DEV),
        to_dev(pr["kept_tok_off"], DEV), torch.from_numpy(pr["kept_tok_off"]),
        to_dev(pr["adv"].astype(np.float32), DEV),
        ref_logp=to_dev(pb.ref, DEV) if cfg.beta else None,
        seq_index=to_dev(pr["kept_traj"].astype(np.int32), DEV),
        row_index=to_dev(pb.src.astype(np.int32), DEV), algo=cfg.algo, norm=cfg.norm,
        eps_low=cfg.eps_low, eps_high=cfg.eps_high, beta=cfg.beta, need_dhidden=backward,
        need_dW=backward, slab_tokens=slab, status=status, need_entropy=True).run()


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("slab", [0, 150])
@pytest.mark.parametrize("backward", [True, False])
def test_entropy_matches_oracle(fr, case, slab, backward):
    c, kw = CASES[case]
    pb = Problem(c, DEV, **kw)
    want = oracle.token_entropy(pb.H64[pb.src], pb.W64)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    call = _call(fr, pb, backward=backward, slab=slab, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    T = len(pb.src)
    got = call.entropy[:T].double().cpu().numpy()
    assert np.abs(got - want).max() < ENT_ATOL, np.abs(got - want).max()
    s = float(call.entropy_sum.item())
    assert abs(s - want.sum()) <= 1e-4 * abs(want.sum()), (s, want.sum())
    # the log-probs of the same call are unchanged by the extra accumulator
    assert np.abs(call.logp[:T].double().cpu().numpy() - pb.logp_exact).max() < LOGP_ATOL


def test_entropy_on_the_shifted_path(fr):
    """Logits far outside exp's float range (rows re-evaluated with a per-row shift)."""
    pb = Problem(3, DEV, Q=3, len_range=(20, 60), V=700, d=64, h_std=40.0, w_std=0.2)
    want = oracle.token_entropy(pb.H64[pb.src], pb.W64)
    call = _call(fr, pb, backward=True)
    torch.cuda.synchronize()
    assert call.stats[1].item() > 0
    T = len(pb.src)
    got = call.entropy[:T].double().cpu().numpy()
    err = np.abs(got - want).max()
    print(f"shifted-path entropy max error {err:.3e}")
    assert err < ENT_ATOL, err
