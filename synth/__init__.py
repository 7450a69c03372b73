"""Seeded synthetic GRPO rollouts shaped like the paper's workloads.

This module draws inputs only: it holds none of the method's arithmetic (no
advantage, pruning, log-softmax or loss).  Both the oracle-side tests and the GPU
path's tests and benchmark use it, so the two sides see the same inputs.

The paper trains Qwen2.5-VL-7B / Qwen3-VL-8B on Geometry3K and GeoQA8K-R1V with
G_1 = 8 rollouts per question and tau = 0.8 (Sec. 4.1).  Those datasets and weights
are not available, so five synthetic workloads stand in for them (LM-head shapes of
Qwen2.5-1.5B and Qwen2.5-VL-7B; uniform token ids; Gaussian hidden states and
weights; Bernoulli rewards).  See ``CONFIGS``.

Random streams (numpy PCG64, ``SeedSequence([seed, stream])``):
  0 prompt success rates and group sizes, 1 lengths, 2 rewards, 3 token ids,
  4 old-logp noise, 5 ref-logp noise.
Dense tensors (hidden states, weights) come from a seeded ``torch.Generator`` on
the device that will hold them, in fixed-size chunks, so a run is reproducible on
one device type.
"""
from dataclasses import dataclass, field
import math

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    Q: int
    G: tuple              # possible group sizes (one drawn per prompt)
    len_lo: int
    len_hi: int
    d: int
    V: int
    dtype: str            # "f32" or "bf16"
    algo: str             # "grpo" | "dapo" | "gspo"
    norm: str             # "seq_mean_token_mean" | "token_mean"
    eps_low: float
    eps_high: float
    beta: float
    keep_ratio: float
    drop_uniform: bool
    format_reward: float  # weight of the Bernoulli(0.9) format reward (0 = none)
    seed: int
    tau_num: int = 4      # tau = 0.8 (Sec. 4.1)
    tau_den: int = 5
    ngram_n: int = 1


CONFIGS = {
    1: Workload("tiny_grpo_f32", 4, (8,), 16, 64, 256, 4096, "f32", "grpo",
                "seq_mean_token_mean", 0.2, 0.2, 0.0, 0.5, False, 0.0, 20261),
    2: Workload("qwen2.5-1.5b_grpo_bf16", 32, (8,), 64, 512, 1536, 151936, "bf16",
                "grpo", "token_mean", 0.2, 0.2, 0.0, 0.5, False, 0.0, 20262),
    3: Workload("qwen2.5-vl-7b_grpo_kl_bf16", 64, (8,), 128, 1024, 3584, 152064,
                "bf16", "grpo", "seq_mean_token_mean", 0.2, 0.2, 0.04, 0.5, False,
                0.1, 20263),
    4: Workload("qwen2.5-vl-7b_dapo_bf16", 64, (16,), 128, 2048, 3584, 152064, "bf16",
                "dapo", "token_mean", 0.2, 0.28, 0.0, 0.5, True, 0.0, 20264),
    5: Workload("qwen2.5-vl-7b_gspo_bf16", 128, (8, 12, 16), 256, 2048, 3584, 152064,
                "bf16", "gspo", "seq_mean_token_mean", 3e-4, 4e-4, 0.0, 0.4, False,
                0.0, 20265),
}

# old/ref log-prob noise: old = new + N(0, 0.05), ref = new + N(0, 0.05)
NOISE_SD = 0.05
# keep token ratios exp(-noise) (and GSPO sequence ratios) this far from a clip
# edge, in log space, so that rounding differences cannot flip a clip decision
TOKEN_EDGE_MARGIN = 1e-4
SEQ_EDGE_MARGIN = 2e-5


def _rng(seed, stream):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, stream])))


@dataclass
class Rollouts:
    cfg: Workload
    group_off: np.ndarray      # int32[Q+1]
    traj_tok_off: np.ndarray   # int64[N+1]
    lengths: np.ndarray        # int64[N]
    rewards: np.ndarray        # float32[N]
    token_ids: np.ndarray      # int32[T_total]
    old_noise: np.ndarray      # float64[T_total]
    ref_noise: np.ndarray      # float64[T_total]
    extra: dict = field(default_factory=dict)

    @property
    def N(self):
        return int(self.group_off[-1])

    @property
    def T_total(self):
        return int(self.traj_tok_off[-1])


def _far_from_edges(v, lo_edge, hi_edge, margin):
    return (np.abs(v - lo_edge) >= margin) & (np.abs(v - hi_edge) >= margin)


def make_rollouts(cfg, seed=None, Q=None, len_range=None, G=None, V=None):
    """Draw the integer/structural part of a workload plus the log-prob noise.

    Optional overrides (Q, len_range, G, V) shrink a workload for small tests while
    keeping its distributions.
    """
    seed = cfg.seed if seed is None else seed
    Q = cfg.Q if Q is None else Q
    lo, hi = (cfg.len_lo, cfg.len_hi) if len_range is None else len_range
    Gs = cfg.G if G is None else tuple(G)
    V = cfg.V if V is None else V
    r0 = _rng(seed, 0)
    p = r0.uniform(0.0, 1.0, size=Q)
    gq = r0.choice(np.asarray(Gs), size=Q) if len(Gs) > 1 else np.full(Q, Gs[0])
    group_off = np.zeros(Q + 1, dtype=np.int32)
    group_off[1:] = np.cumsum(gq)
    N = int(group_off[-1])
    lengths = _rng(seed, 1).integers(lo, hi + 1, size=N).astype(np.int64)
    traj_tok_off = np.zeros(N + 1, dtype=np.int64)
    traj_tok_off[1:] = np.cumsum(lengths)
    r2 = _rng(seed, 2)
    pp = np.repeat(p, gq)
    rewards = (r2.uniform(size=N) < pp).astype(np.float32)
    if cfg.format_reward:
        fmt = (r2.uniform(size=N) < 0.9).astype(np.float32)
        rewards = (rewards + np.float32(cfg.format_reward) * fmt).astype(np.float32)
    T = int(traj_tok_off[-1])
    token_ids = _rng(seed, 3).integers(0, V, size=T).astype(np.int32)

    r4 = _rng(seed, 4)
    old_noise = r4.normal(0.0, NOISE_SD, size=T)
    lo_e, hi_e = math.log1p(-cfg.eps_low), math.log1p(cfg.eps_high)
    if cfg.algo == "gspo":
        # sequence log-ratio mean(x - o) = -mean(noise); keep it off the clip edges
        for i in range(N):
            a, b = int(traj_tok_off[i]), int(traj_tok_off[i + 1])
            while b > a and not _far_from_edges(-old_noise[a:b].mean(), lo_e, hi_e,
                                                SEQ_EDGE_MARGIN):
                old_noise[a:b] = r4.normal(0.0, NOISE_SD, size=b - a)
    else:
        bad = ~_far_from_edges(-old_noise, lo_e, hi_e, TOKEN_EDGE_MARGIN)
        while bad.any():
            old_noise[bad] = r4.normal(0.0, NOISE_SD, size=int(bad.sum()))
            bad = ~_far_from_edges(-old_noise, lo_e, hi_e, TOKEN_EDGE_MARGIN)
    ref_noise = _rng(seed, 5).normal(0.0, NOISE_SD, size=T)
    return Rollouts(cfg, group_off, traj_tok_off, lengths, rewards, token_ids,
                    old_noise, ref_noise, extra={"V": V, "seed": seed})


def make_dense(cfg, T_rows, device="cpu", seed=None, d=None, V=None, chunk=1 << 24,
               w_std=0.02, h_std=1.0):
    """Hidden states H[T_rows, d] ~ N(0, h_std^2) and weights W[V, d] ~ N(0, w_std^2),
    drawn in float32 from a seeded torch generator on ``device`` and rounded
    (round-to-nearest-even) to the workload dtype."""
    import torch
    seed = cfg.seed if seed is None else seed
    d = cfg.d if d is None else d
    V = cfg.V if V is None else V
    dt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    gen = torch.Generator(device=device)

    def draw(rows, std, sub):
        gen.manual_seed(seed * 1000 + sub)
        out = torch.empty((rows, d), dtype=dt, device=device)
        flat = out.view(-1)
        step = max(d, (chunk // d) * d)
        for a in range(0, flat.numel(), step):
            b = min(flat.numel(), a + step)
            flat[a:b] = (torch.randn(b - a, generator=gen, device=device,
                                     dtype=torch.float32) * std).to(dt)
        return out

    return draw(T_rows, h_std, 7), draw(V, w_std, 8)


def continuous_rewards(group_off, seed, scale=1.2, near=5e-5):
    """Continuous rewards shaped like the grounding task's (an IoU-like and a centre-in
    score): per question a few base values ~ U(0, scale); each rollout repeats a base
    value exactly (probability 0.4: the same box twice), repeats it up to +-``near``
    (0.3: a box a few pixels off), or draws a fresh U(0, scale) value.  Exact and near
    repeats make advantage gaps on both sides of 1e-4.  float32[N]."""
    rng = _rng(seed, 6)
    off = np.asarray(group_off, dtype=np.int64)
    out = np.zeros(int(off[-1]), dtype=np.float32)
    for q in range(len(off) - 1):
        a, b = int(off[q]), int(off[q + 1])
        base = rng.uniform(0.0, scale, size=4)
        for i in range(a, b):
            k = int(rng.integers(0, 4))
            u = rng.uniform()
            if u < 0.4:
                out[i] = base[k]
            elif u < 0.7:
                out[i] = base[k] + rng.uniform(-near, near)
            else:
                out[i] = rng.uniform(0.0, scale)
    return out


def plant_duplicates(ro, p_copy=0.6, p_mutate=0.15, seed=7):
    """Test-only structure: inside each question, overwrite some trajectories with a
    near-copy of the question's first trajectory (each position re-drawn with probability
    p_mutate), so n-gram Jaccard distances fall below tau and MDAP has work to do.
    Modifies ``ro.token_ids`` in place."""
    rng = _rng(seed, 99)
    V = int(ro.extra["V"])
    for q in range(len(ro.group_off) - 1):
        a, b = int(ro.group_off[q]), int(ro.group_off[q + 1])
        base = ro.token_ids[ro.traj_tok_off[a]:ro.traj_tok_off[a + 1]].copy()
        for i in range(a + 1, b):
            if rng.uniform() >= p_copy or len(base) == 0:
                continue
            s0, s1 = int(ro.traj_tok_off[i]), int(ro.traj_tok_off[i + 1])
            L = s1 - s0
            t = np.resize(base, L)
            m = rng.uniform(size=L) < p_mutate
            t[m] = rng.integers(0, V, size=int(m.sum()))
            ro.token_ids[s0:s1] = t
    return ro


def skew_tokens(ro, frac, token=0, seed=11):
    """Test-only structure: a head-heavy token distribution, as in real text where a few ids
    (spaces, punctuation, end of text) fill a large share of the positions.  Each position
    becomes ``token`` with probability ``frac`` (1.0: every position).  Modifies
    ``ro.token_ids`` in place."""
    rng = _rng(seed, 98)
    m = rng.uniform(size=ro.token_ids.shape[0]) < frac
    ro.token_ids[m] = token
    return ro
