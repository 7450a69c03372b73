"""Planted mistakes in the oracle are caught by its pins.

Each case copies the source of ``oracle/loss.py``, plants one plausible mistake (a plain
text substitution, asserted to apply), loads the copy as a separate module on the CPU and
runs the hand-derived fixture checks against it: every mutant must fail at least one of
them, while the unmodified source passes all of them."""
import importlib.util
import os
import sys

import pytest

from tests.test_oracle_loss_golden import check_gspo_golden, check_kl_golden

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LOSS_SRC = os.path.join(ROOT, "oracle", "loss.py")

MUTANTS = {
    "gspo_sum_for_mean": ("s = np.exp(np.sum(x[a:b] - o[a:b]) / L)",
                          "s = np.exp(np.sum(x[a:b] - o[a:b]))"),
    "gspo_mean_of_token_ratios": ("s = np.exp(np.sum(x[a:b] - o[a:b]) / L)",
                                  "s = np.mean(np.exp(x[a:b] - o[a:b]))"),
    "gspo_first_token_ratio": ("s = np.exp(np.sum(x[a:b] - o[a:b]) / L)",
                               "s = np.exp(x[a] - o[a])"),
    "k3_reversed": ("k3 = np.exp(f - x) - (f - x) - 1.0\n        dk3 = 1.0 - np.exp(f - x)",
                    "k3 = np.exp(x - f) - (x - f) - 1.0\n        dk3 = np.exp(x - f) - 1.0"),
    "kl_gradient_sign": ("g += beta * w * dk3", "g -= beta * w * dk3"),
    "gspo_clip_exclusive_edge": ("(Ai >= 0 and s <= hi) or (Ai < 0 and s >= lo)",
                                 "(Ai >= 0 and s < hi) or (Ai < 0 and s > lo)"),
}


def _load_variant(src, tag):
    name = f"_oracle_loss_{tag}"
    spec = importlib.util.spec_from_loader(name, loader=None)
    mod = importlib.util.module_from_spec(spec)
    exec(compile(src, f"<{name}>", "exec"), mod.__dict__)
    sys.modules.pop(name, None)
    return mod


def _fails(fn):
    try:
        fn()
    except AssertionError:
        return True
    return False


def test_unmodified_source_passes():
    mod = _load_variant(open(LOSS_SRC).read(), "orig")
    check_gspo_golden(mod.policy_loss)
    check_kl_golden(mod.policy_loss)


@pytest.mark.parametrize("name", list(MUTANTS))
def test_planted_mistake_is_caught(name):
    old, new = MUTANTS[name]
    src = open(LOSS_SRC).read()
    assert src.count(old) == 1, f"mutation site of {name} not found in oracle/loss.py"
    mod = _load_variant(src.replace(old, new), name)
    pl = mod.policy_loss
    assert _fails(lambda: check_gspo_golden(pl)) or _fails(lambda: check_kl_golden(pl)), name
