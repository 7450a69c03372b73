"""Plain fp64 CPU oracle for the FastRL GRPO-step hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this package.
The product path (``paper_2609_36932_amd``) never imports it and shares no code,
headers, tables or helpers with it.

Each module follows one part of the paper (arXiv 2609.36932, "Learn from the Gap:
Differential-Aware Advantage Pruning with Adaptive Rollout Sampling for GRPO"):

* ``advantage`` -- group-normalised advantage (Sec. 3.2, Eq. advantage)
* ``mdap``      -- advantage partition, n-gram Jaccard distance, greedy de-redundancy
                   (Sec. 3.2, Eq. grouping and the S'_k definition; Alg. 1 Phase 2),
                   the keep-ratio budget, and stream compaction of kept tokens
* ``lmhead``    -- LM-head log-probabilities and their backward (Sec. 3.2, the
                   post-pruning evaluation paragraph; Sec. 3.1 gradient)
* ``loss``      -- GRPO / DAPO / GSPO clipped surrogate and its per-token gradient
                   coefficient (Sec. 3.1, Eq. 1, Eq. grad, clipping indicator)
* ``ars``       -- adaptive rollout sampling controller (Sec. 3.3; Alg. 1 Phase 1)
* ``optim``     -- the AdamW step on W consuming dW (Sec. 4.1 hyper-parameters)
* ``pipeline``  -- one hot-path step end to end, in the order of Alg. 1

Everything is float64 (rewards, hidden states and weights are read as the exact
float64 values of their stored float32 / bfloat16 bits).  Integer decisions
(classes, pruning, budget, compaction) are exact.
"""
from .advantage import group_advantage
from .mdap import (ngram_set, jaccard_counts, theta_below_tau, greedy_mdap_class,
                   budget_keep, prune_prompt, prune_batch, compact, continuous_classes,
                   visit_order, dp_align_fill)
from .lmhead import token_logprob, lmhead_backward, lmhead_dW_rows, logits, token_entropy
from .loss import policy_loss, token_weights
from .ars import ARSController
from .optim import adamw_step
from .pipeline import hot_path_step

__all__ = [
    "group_advantage", "ngram_set", "jaccard_counts", "theta_below_tau",
    "greedy_mdap_class", "budget_keep", "prune_prompt", "prune_batch", "compact",
    "continuous_classes", "visit_order", "dp_align_fill",
    "token_logprob", "lmhead_backward", "lmhead_dW_rows", "logits", "token_entropy", "policy_loss",
    "token_weights",
    "ARSController", "hot_path_step", "adamw_step",
]
