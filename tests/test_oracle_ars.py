"""Pins for the oracle's adaptive rollout sampling controller (Sec. 3.3, Alg. 1
Phase 1): hand-derived sequences, range and no-early-adjustment properties."""
import json
import os

import numpy as np
import pytest

from oracle import ARSController


def test_golden_sequences(golden_dir):
    d = json.load(open(os.path.join(golden_dir, "ars_sequence.json")))
    for run in d["runs"]:
        c = ARSController(run["G"], run["M"], run["E"])
        ns = []
        for counts in run["steps"]:
            ns.append(c.next_n())
            c.observe(counts)
        assert ns == run["n_before_step"]
        assert c.next_n() == run["n_after"]
        assert c.G_ref == pytest.approx(run["G_ref"], abs=1e-12)
        assert c.G_t == pytest.approx(run["G_t_final"], abs=1e-12)


@pytest.mark.parametrize("seed", range(20))
def test_range_and_no_early_adjustment(seed):
    rng = np.random.default_rng(seed)
    G = int(rng.choice([4, 8, 16]))
    E = int(rng.integers(1, 5))
    M = E * int(rng.integers(1, 6))
    c = ARSController(G, M, E)
    for step in range(M + 3):
        n = c.next_n()
        assert 2 <= n <= G
        if step < E:
            assert n == G  # nothing set before the first epoch ends
        counts = rng.integers(1, n + 1, size=int(rng.integers(1, 6)))
        c.observe(counts)


def test_first_boundary_trigger_needs_alpha_above_half():
    # at the first boundary G'_t < G'_ref  <=>  alpha > 1/2 (when max > mean)
    for M, E in [(10, 2), (4, 2), (3, 2)]:
        c = ARSController(8, M, E)
        for _ in range(E):
            c.observe([2, 6])
        alpha = E / M
        assert (c.G_t < c.G_ref) == (alpha > 0.5)
        # triggered: n = max(round(min(G - (G'_ref - G'_t), G)), 2)
        want = max(round(min(8 - (c.G_ref - c.G_t), 8)), 2) if alpha > 0.5 else 8
        assert c.next_n() == want
