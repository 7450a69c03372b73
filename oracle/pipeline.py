"""Oracle: one hot-path step end to end, in the order of Alg. 1 (test
infrastructure only; see oracle/__init__):

  rewards -> advantages (Eq. advantage) -> MDAP pruning + budget (Sec. 3.2,
  Alg. 1 Phase 2) -> compaction of kept tokens -> LM-head log-probs of the kept
  tokens (Sec. 3.2, post-pruning evaluation) -> clipped surrogate loss and per-token
  gradient coefficient (Sec. 3.1) -> LM-head backward to dH and dW.
"""
import numpy as np

from .advantage import group_advantage
from .mdap import prune_batch, compact, dp_align_fill
from .lmhead import token_logprob, lmhead_backward
from .loss import policy_loss


def hot_path_step(rewards, group_off, token_ids, traj_tok_off, *, H=None, W=None,
                  old_logp=None, ref_logp=None, algo="grpo",
                  norm="seq_mean_token_mean", eps_low=0.2, eps_high=0.2, beta=0.0,
                  ngram_n=1, tau_num=4, tau_den=5, keep_ratio=0.0,
                  drop_uniform=False, std_ddof=1, adv_eps=1e-6, group_eps=0.0, dp_align=1,
                  lmhead=True):
    """``group_eps`` > 0: continuous-reward groups |A_i - A_j| < group_eps (appendix on
    the grounding task) instead of bit-equal reward classes.  ``dp_align`` > 1: Alg. 1's
    fill of the kept set up to a multiple of the data-parallel divisor."""
    out = {}
    adv, cls, valid = group_advantage(rewards, group_off, ddof=std_ddof, eps=adv_eps,
                                      drop_uniform=drop_uniform)
    out.update(adv=adv, class_id=cls, group_valid=valid)
    # the pruning step sees the float32 advantages the advantage step outputs
    adv32 = adv.astype(np.float32)
    keep, counts, used = prune_batch(token_ids, traj_tok_off, rewards, group_off, cls, valid,
                                     ngram_n=ngram_n, tau_num=tau_num, tau_den=tau_den,
                                     keep_ratio=keep_ratio, adv=adv32, group_eps=group_eps,
                                     return_classes=True)
    keep, added = dp_align_fill(keep, adv32, group_off, valid, dp_align)
    out.update(keep_mask=keep, mdap_count=counts, prune_class=used, dp_added=added)
    kept, koff, src = compact(keep, traj_tok_off)
    out.update(kept_traj=kept, kept_tok_off=koff, tok_src=src)
    if not lmhead:
        return out
    y = np.asarray(token_ids, dtype=np.int64)[src]
    Hk = np.asarray(H, dtype=np.float64)[src]
    logp, lse = token_logprob(Hk, W, y)
    ref = None if ref_logp is None else np.asarray(ref_logp, dtype=np.float64)[src]
    loss, g, info = policy_loss(logp, np.asarray(old_logp, dtype=np.float64)[src], ref,
                                koff, adv[kept], algo=algo, norm=norm,
                                eps_low=eps_low, eps_high=eps_high, beta=beta)
    dH, dW = lmhead_backward(Hk, W, y, lse, g)
    out.update(logp=logp, lse=lse, loss=loss, g=g, dH=dH, dW=dW, info=info)
    return out
