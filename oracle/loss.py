"""Oracle: GRPO / DAPO / GSPO clipped surrogate loss and its per-token gradient
coefficient g_t = dL/dlogp_t (test infrastructure only; see oracle/__init__).

Paper, Sec. 3.1: Eq. (1) is the GRPO objective J (maximised); the loss here is
L = -J.  The gradient expansion and Eq. (grad) give, per token,
    [c_t * rho_t * A_i + beta * (pi_ref / pi_theta - 1)] * grad log pi_theta
with the clipping indicator c_t = 1[A>=0] 1[rho<=1+eps] + 1[A<0] 1[rho>=1-eps]
(inclusive edges).  With x = logp, o = old logp, f = ref logp, rho = exp(x - o):

* token objectives (GRPO, DAPO):
    l_t = -min(rho A, clip(rho, 1-eps_low, 1+eps_high) A) + beta * k3_t
    k3_t = exp(f - x) - (f - x) - 1        (the KL estimator whose gradient is the
                                            paper's beta (pi_ref/pi_theta - 1) term)
    g_t = w_t * (-c_t rho_t A + beta * (1 - exp(f - x)))
* sequence objective (GSPO, sequence ratio = exp(mean token log-ratio)):
    s_i = exp((1/L_i) sum_t (x_t - o_t))
    l_i = -min(s_i A, clip(s_i, 1-eps_low, 1+eps_high) A)
    g_t = W_i * (-c_i s_i A / L_i) + beta * w_t * (1 - exp(f - x))

Normalisation (Eq. 1 averages over the G rollouts and over each rollout's tokens;
after pruning G becomes the number S of kept sequences):
* "seq_mean_token_mean": w_t = 1 / (S * L_i)
* "token_mean":          w_t = 1 / T   (T = all kept tokens; DAPO's token level)
and W_i = sum_{t in i} w_t is the weight of a sequence-level term.
L = sum_t w_t l_t (token objectives) or sum_i W_i l_i + beta sum_t w_t k3_t (GSPO).
A sequence with no tokens contributes nothing (it still counts in S).
"""
import numpy as np

ALGOS = ("grpo", "dapo", "gspo")
NORMS = ("seq_mean_token_mean", "token_mean")


def token_weights(seq_off, norm):
    off = np.asarray(seq_off, dtype=np.int64)
    S = len(off) - 1
    T = int(off[-1]) - int(off[0]) if S >= 0 else 0
    w = np.zeros(T, dtype=np.float64)
    base = int(off[0])
    for i in range(S):
        a, b = int(off[i]) - base, int(off[i + 1]) - base
        L = b - a
        if L == 0:
            continue
        if norm == "seq_mean_token_mean":
            w[a:b] = 1.0 / (S * L)
        elif norm == "token_mean":
            w[a:b] = 1.0 / T
        else:
            raise ValueError(norm)
    return w


def policy_loss(logp, old_logp, ref_logp, seq_off, adv, algo="grpo",
                norm="seq_mean_token_mean", eps_low=0.2, eps_high=0.2, beta=0.0):
    """Return (loss float, g float64[T], info dict)."""
    if algo not in ALGOS:
        raise ValueError(algo)
    x = np.asarray(logp, dtype=np.float64)
    o = np.asarray(old_logp, dtype=np.float64)
    off = np.asarray(seq_off, dtype=np.int64)
    base = int(off[0])
    S = len(off) - 1
    A = np.asarray(adv, dtype=np.float64)
    w = token_weights(off, norm)
    T = len(x)
    g = np.zeros(T, dtype=np.float64)
    loss = 0.0
    clipped = 0
    if beta != 0.0:
        f = np.asarray(ref_logp, dtype=np.float64)
        k3 = np.exp(f - x) - (f - x) - 1.0
        dk3 = 1.0 - np.exp(f - x)
        loss += float(np.sum(w * k3)) * beta
        g += beta * w * dk3
    lo, hi = 1.0 - eps_low, 1.0 + eps_high
    for i in range(S):
        a, b = int(off[i]) - base, int(off[i + 1]) - base
        L = b - a
        if L == 0:
            continue
        Ai = A[i]
        if algo == "gspo":
            s = np.exp(np.sum(x[a:b] - o[a:b]) / L)
            sur = min(s * Ai, min(max(s, lo), hi) * Ai)
            c = 1.0 if ((Ai >= 0 and s <= hi) or (Ai < 0 and s >= lo)) else 0.0
            Wi = float(np.sum(w[a:b]))
            loss += -Wi * sur
            g[a:b] += Wi * (-c * s * Ai / L)
            clipped += int(c == 0.0) * L
        else:
            rho = np.exp(x[a:b] - o[a:b])
            sur = np.minimum(rho * Ai, np.clip(rho, lo, hi) * Ai)
            if Ai >= 0:
                c = (rho <= hi).astype(np.float64)
            else:
                c = (rho >= lo).astype(np.float64)
            loss += float(np.sum(-w[a:b] * sur))
            g[a:b] += w[a:b] * (-c * rho * Ai)
            clipped += int(np.sum(c == 0.0))
    return loss, g, {"clipped_tokens": clipped, "weights": w}
