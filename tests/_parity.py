"""Shared helpers of the GPU parity tests: build one seeded problem, run the oracle and
the HIP path (through the C ABI) on the same inputs, compare with the stated bars:
pruning masks / indices bit-exact, log-probs 2e-3 absolute, loss and gradients 1e-2
relative (bf16 inputs, fp32 accumulate): for gradients both the whole-matrix relative
Frobenius error and the largest per-row relative error."""
import dataclasses

import numpy as np
import torch

import oracle
from synth import CONFIGS, make_rollouts, make_dense, plant_duplicates, skew_tokens

LOGP_ATOL = 2e-3
REL = 1e-2
# log-prob error assumed when bounding how far g may move per row: the synthetic inputs keep
# every token (and GSPO sequence) ratio at least this far from a clip edge in log space, so
# no clip decision flips within it (measured GPU log-prob errors are ~1e-5)
G_LOGP_EPS = 1e-4
# unit roundoff of the exp-logit operand of the backward GEMMs: bfloat16 (8 significant bits)
# and float32
BF16_U = 2.0 ** -8
FP32_U = 2.0 ** -24


def rel_fro(a, b):
    nb = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (nb if nb > 0 else 1.0)


def to_dev(x, dev, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(dev)


class Problem:
    """Seeded problem: rollouts, oracle pruning, dense tensors and old/ref log-probs built
    from the oracle's exact log-probs of the kept tokens (+ the seeded noise)."""

    def __init__(self, cfg_id, dev, *, Q=None, len_range=None, G=None, V=None, d=None,
                 dtype=None, seed=None, h_std=1.0, w_std=0.02, ngram_n=None, keep_ratio=None,
                 tau=None, vocab_ids=None, planted=None, skew=None):
        base = CONFIGS[cfg_id]
        self.cfg = base
        self.V = V or base.V
        self.d = d or base.d
        self.dtype = dtype or base.dtype
        self.fold_u = FP32_U if self.dtype == "f32" else BF16_U
        self.keep_ratio = base.keep_ratio if keep_ratio is None else keep_ratio
        self.tau = (base.tau_num, base.tau_den) if tau is None else tau
        self.ngram_n = base.ngram_n if ngram_n is None else ngram_n
        ro = make_rollouts(base, seed=seed, Q=Q, len_range=len_range, G=G, V=vocab_ids or self.V)
        if planted is not None:
            plant_duplicates(ro, **planted)
        if skew is not None:
            skew_tokens(ro, skew)
        self.ro = ro
        self.dev = dev
        pr = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                                  lmhead=False, ngram_n=self.ngram_n, tau_num=self.tau[0],
                                  tau_den=self.tau[1], keep_ratio=self.keep_ratio,
                                  drop_uniform=base.drop_uniform)
        self.pr = pr
        self.src = pr["tok_src"]
        self.max_group = int(np.diff(ro.group_off).max())
        self.max_len = int(ro.lengths.max())
        cfg_dt = dataclasses.replace(base, dtype=self.dtype)
        H, W = make_dense(cfg_dt, ro.T_total, device="cpu", d=self.d, V=self.V,
                          seed=seed, h_std=h_std, w_std=w_std)
        self.H, self.W = H, W
        self.H64 = H.double().numpy()
        self.W64 = W.double().numpy()
        y = ro.token_ids[self.src].astype(np.int64)
        self.y = y
        lp, lse = oracle.token_logprob(self.H64[self.src], self.W64, y)
        self.logp_exact, self.lse_exact = lp, lse
        old = np.full(ro.T_total, np.nan)
        ref = np.full(ro.T_total, np.nan)
        old[self.src] = lp + ro.old_noise[self.src]
        ref[self.src] = lp + ro.ref_noise[self.src]
        self.old = old.astype(np.float32)
        self.ref = ref.astype(np.float32)
        # poison every pruned row: the HIP path must never read it
        Hp = H.clone()
        pruned = np.ones(ro.T_total, dtype=bool)
        pruned[self.src] = False
        Hp[torch.from_numpy(pruned)] = float("nan")
        self.H_poisoned = Hp

    def scale_hidden(self, rows, factor):
        """Multiply the hidden rows `rows` (indices into the full batch) by `factor` (a power of
        two, exact in bf16) and redo everything built from H: the oracle's log-probs and
        log-sum-exps of the kept tokens, the old / ref log-probs, the poisoned copy."""
        H = self.H.clone()
        H[torch.as_tensor(rows, dtype=torch.long)] *= factor
        self.H = H
        self.H64 = H.double().numpy()
        lp, lse = oracle.token_logprob(self.H64[self.src], self.W64, self.y)
        self.logp_exact, self.lse_exact = lp, lse
        ro = self.ro
        old = np.full(ro.T_total, np.nan)
        ref = np.full(ro.T_total, np.nan)
        old[self.src] = lp + ro.old_noise[self.src]
        ref[self.src] = lp + ro.ref_noise[self.src]
        self.old = old.astype(np.float32)
        self.ref = ref.astype(np.float32)
        Hp = H.clone()
        pruned = np.ones(ro.T_total, dtype=bool)
        pruned[self.src] = False
        Hp[torch.from_numpy(pruned)] = float("nan")
        self.H_poisoned = Hp

    def oracle_loss(self):
        base = self.cfg
        kept = self.pr["kept_traj"]
        loss, g, info = oracle.policy_loss(
            self.logp_exact, self.old[self.src].astype(np.float64),
            self.ref[self.src].astype(np.float64) if base.beta else None,
            self.pr["kept_tok_off"], self.pr["adv"][kept], algo=base.algo, norm=base.norm,
            eps_low=base.eps_low, eps_high=base.eps_high, beta=base.beta)
        dH, dW = oracle.lmhead_backward(self.H64[self.src], self.W64, self.y, self.lse_exact, g)
        return dict(loss=loss, g=g, dH=dH, dW=dW, clipped=info["clipped_tokens"],
                    dg=self.g_dev())

    def g_dev(self, eps=G_LOGP_EPS):
        """g_deviation of this problem's oracle g under log-prob errors of eps."""
        base = self.cfg
        kept = self.pr["kept_traj"]
        return g_deviation(self.logp_exact, self.old[self.src].astype(np.float64),
                           self.ref[self.src].astype(np.float64) if base.beta else None,
                           self.pr["kept_tok_off"], self.pr["adv"][kept], eps=eps,
                           algo=base.algo, norm=base.norm, eps_low=base.eps_low,
                           eps_high=base.eps_high, beta=base.beta)

    def run_gpu(self, fr, slab_tokens=0, dhidden_dtype=None, status=None, poisoned=True):
        dev = self.dev
        ro = self.ro
        base = self.cfg
        H = (self.H_poisoned if poisoned else self.H).to(dev)
        W = self.W.to(dev)
        old = to_dev(self.old, dev)
        ref = to_dev(self.ref, dev) if base.beta else None
        return fr.hot_path_step(
            to_dev(ro.rewards, dev), to_dev(ro.group_off, dev), to_dev(ro.token_ids, dev),
            to_dev(ro.traj_tok_off, dev), H, W, old, ref, V=self.V, max_group=self.max_group,
            max_len=self.max_len, algo=base.algo, norm=base.norm, eps_low=base.eps_low,
            eps_high=base.eps_high, beta=base.beta, ngram_n=self.ngram_n, tau=self.tau,
            keep_ratio=self.keep_ratio, drop_uniform=base.drop_uniform,
            slab_tokens=slab_tokens, status=status, dhidden_dtype=dhidden_dtype)


def fold_bounds(H, W, y, g, u=BF16_U):
    """Frobenius bounds of what the one-hot fold adds to the error of dhidden and of dW.  The
    backward GEMMs take the one-hot term of dZ from the exp-logit operand: its label entry
    E[t][y_t] - exp(lse_t - s_t) is rounded once to the operand's precision (unit roundoff u,
    as in a dlogits operand of that type), and with E[t][y_t]'s own rounding the entry times
    c_t moves by at most u |g_t| (|p_ty - 1| + p_ty = 1): u |g_t| ||W_{y_t}|| in dhidden row t,
    sum_{t: y_t = v} u |g_t| ||H_t|| in dW row v."""
    H = np.asarray(H, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    a = u * np.abs(np.asarray(g, dtype=np.float64))
    bH = a * np.linalg.norm(W[y], axis=1)
    bW = np.zeros(W.shape[0])
    np.add.at(bW, y, a * np.linalg.norm(H, axis=1))
    return float(np.sqrt((bH ** 2).sum())), float(np.sqrt((bW ** 2).sum()))


def soft_excess(gpu, ref, part, bound, rel=REL):
    """The softmax part alone (the reference minus its one-hot part): ||gpu - ref|| against
    rel ||ref - part|| + bound (fold_bounds), as a ratio scaled by rel (<= rel passes)."""
    num = np.linalg.norm(np.asarray(gpu, dtype=np.float64) - ref)
    den = rel * np.linalg.norm(ref - part) + bound
    return rel * (num / den if den > 0 else (0.0 if num == 0 else np.inf))


def onehot_parts(H, W, y, g):
    """The sparse parts of the LM-head gradient: g_t W[y_t] (dH) and the scatter of
    g_t H_t onto row y_t (dW)."""
    dH1 = g[:, None] * W[y]
    dW1 = np.zeros_like(W)
    np.add.at(dW1, y, g[:, None] * H)
    return dH1, dW1


def row_rel(a, b, part=None):
    """Largest per-row relative error max_r ||a_r - b_r|| / ||b_r|| (rows whose reference is
    exactly zero must be exactly zero: they count as 0 or inf).  With `part` (the one-hot
    part of the reference rows) the denominator is ||part_r|| + ||b_r - part_r||, the norms
    of the row's two parts: within a factor sqrt(2) of ||b_r|| when they do not cancel, and
    the scale of the float32 rounding when they do (a token whose probability is ~1)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    num = np.linalg.norm(a - b, axis=1)
    if part is None:
        den = np.linalg.norm(b, axis=1)
    else:
        part = np.asarray(part, dtype=np.float64)
        den = np.linalg.norm(part, axis=1) + np.linalg.norm(b - part, axis=1)
    r = np.where(den > 0, num / np.where(den > 0, den, 1.0), np.where(num > 0, np.inf, 0.0))
    return float(r.max()) if len(r) else 0.0


def g_deviation(logp, old, ref, seq_off, adv, eps=G_LOGP_EPS, **kw):
    """Per token, how far the oracle's g = dL/dlogp moves when every log-prob moves by +-eps:
    max(|g(x + eps) - g(x)|, |g(x - eps) - g(x)|) (for GSPO this is the shift of the sequence
    mean, the worst case of per-token errors of size eps).  Oracle-only quantities."""
    x = np.asarray(logp, dtype=np.float64)
    g0 = oracle.policy_loss(x, old, ref, seq_off, adv, **kw)[1]
    gp = oracle.policy_loss(x + eps, old, ref, seq_off, adv, **kw)[1]
    gm = oracle.policy_loss(x - eps, old, ref, seq_off, adv, **kw)[1]
    return np.maximum(np.abs(gp - g0), np.abs(gm - g0))


def row_tol_excess(gpu, ref, extra, rel):
    """Largest ratio ||gpu_r - ref_r|| / (rel ||ref_r|| + extra_r) over rows (<= 1 passes)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.linalg.norm(gpu - ref, axis=1)
    den = rel * np.linalg.norm(ref, axis=1) + extra
    r = np.where(den > 0, num / np.where(den > 0, den, 1.0), np.where(num > 0, np.inf, 0.0))
    return float(r.max()) if len(r) else 0.0


def check_grads(H, W, y, g_ref, dH_gpu, dW_gpu, dH_ref, dW_ref, rel=REL, dg=None, lse=None,
                u=BF16_U):
    """Whole-gradient relative Frobenius error; the softmax part alone (the one-hot part
    dominates the norm) within rel of its norm plus the bound of the one-hot term's rounding
    in the exp-logit operand (fold_bounds, unit roundoff u); and per row (every token's dhidden
    row, every vocabulary row of dW): ||gpu_r - ref_r|| <= rel ||ref_r|| + e_r, where e_r is
    what a per-token deviation dg of g (g_deviation: the oracle's g under a log-prob error of
    G_LOGP_EPS) moves that row by: dg_t ||W_{y_t} - sum_v p_tv W_v|| for dhidden row t and
    sum_t dg_t |1[y_t = v] - p_tv| ||H_t|| for dW row v.  A row whose g is ill-conditioned (a
    token whose reference log-prob is within ~1e-3 of the current one) thereby gets the
    tolerance the log-prob accuracy implies; every other row is held to rel."""
    out = {}
    T = len(y)
    if dg is None:
        eH, eW = np.zeros(T), np.zeros(W.shape[0])
    else:
        z = np.asarray(H, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
        P = np.exp(z - np.asarray(lse, dtype=np.float64)[:, None])
        A = -P
        A[np.arange(T), y] += 1.0
        eH = np.asarray(dg) * np.linalg.norm(A @ W, axis=1)
        eW = np.abs(A).T @ (np.asarray(dg) * np.linalg.norm(H, axis=1))
    bH, bW = fold_bounds(H, W, y, g_ref, u)
    dH1, dW1 = onehot_parts(H, W, y, g_ref)
    if dH_gpu is not None:
        out["dH"] = rel_fro(dH_gpu, dH_ref)
        out["dH_soft"] = soft_excess(dH_gpu, dH_ref, dH1, bH, rel)
        out["dH_row"] = row_tol_excess(dH_gpu, dH_ref, eH, rel) * rel
    if dW_gpu is not None:
        out["dW"] = rel_fro(dW_gpu, dW_ref)
        out["dW_soft"] = soft_excess(dW_gpu, dW_ref, dW1, bW, rel)
        out["dW_row"] = row_tol_excess(dW_gpu, dW_ref, eW, rel) * rel
    for k, v in out.items():
        assert v <= rel, (k, v, out)
    return out
