"""Oracle: group-relative advantage (test infrastructure only; see oracle/__init__).

Paper: Sec. 3.2, Eq. (advantage): A_i = (r_i - mean{r}) / std{r}, computed over
the G rollouts of one question.  Alg. 1 computes it right after the rewards.

Readings where the paper is silent:
* std uses ``ddof`` (default 1, the sample standard deviation) and ``eps`` is
  added to the denominator (default 1e-6) so an all-equal group gives A = 0; eps is
  a float32 parameter of the library, so the float64 value of float32(eps) is added.
* Advantage classes (Eq. grouping, S_k = {o_i : A_i = a_k}) are taken as classes of
  equal float32 reward value: within a question A is a strictly increasing function
  of r whenever std > 0, and when std = 0 every A is 0 (one class).  Class ids are
  numbered 0, 1, ... in order of first occurrence inside the question.
* a zero denominator (all rewards equal and eps = 0) gives A = 0.
* DAPO-style dropping (``drop_uniform``): a question whose rewards are all equal
  is marked invalid (group_valid = 0).
"""
import math

import numpy as np


def group_advantage(rewards, group_off, ddof=1, eps=1e-6, drop_uniform=False):
    """Return (adv float64[N], class_id int32[N], group_valid uint8[Q]).

    rewards   : float32[N] (read as exact float64)
    group_off : int[Q+1], question q owns trajectories group_off[q]:group_off[q+1]
    """
    r32 = np.asarray(rewards, dtype=np.float32)
    off = np.asarray(group_off, dtype=np.int64)
    Q = len(off) - 1
    N = int(off[-1]) if Q >= 0 else 0
    adv = np.zeros(N, dtype=np.float64)
    cls = np.zeros(N, dtype=np.int32)
    valid = np.ones(Q, dtype=np.uint8)
    for q in range(Q):
        a, b = int(off[q]), int(off[q + 1])
        G = b - a
        if G == 0:
            valid[q] = 0
            continue
        r = [float(x) for x in r32[a:b]]
        m = 0.0
        for x in r:  # index order
            m += x
        m = m / G
        if G - ddof > 0:
            ss = 0.0
            for x in r:  # index order
                ss += (x - m) * (x - m)
            s = math.sqrt(ss / (G - ddof))
        else:
            s = 0.0
        den = s + float(np.float32(eps))
        for i, x in enumerate(r):
            # den == 0 only for an all-equal group with eps == 0: A = 0 (numerator is 0)
            adv[a + i] = (x - m) / den if den > 0 else 0.0
        # classes: equal reward value, numbered by first occurrence
        seen = []
        for i, x in enumerate(r):
            k = None
            for j, y in enumerate(seen):
                if y == x:
                    k = j
                    break
            if k is None:
                seen.append(x)
                k = len(seen) - 1
            cls[a + i] = k
        if drop_uniform and len(seen) == 1:
            valid[q] = 0
    return adv, cls, valid
