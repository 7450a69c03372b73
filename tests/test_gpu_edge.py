"""GPU parity on the edges of what the C ABI accepts: groups of 65 to 256 rollouts (the
selection and pair kernels then loop past one wavefront), zero-length trajectories (through
pruning and the whole loss), a trajectory of max_len = 16384 tokens (a 128 KB n-gram sort in
LDS), trigrams at the largest vocabulary (V = 2^21 - 1: three 21-bit ids fill 63 bits of a
key), and a loss call whose kept sequences are all empty over a NaN-filled workspace.
Pruning results are compared bit for bit with the oracle."""

import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, make_rollouts, plant_duplicates, Rollouts
from tests._parity import Problem, to_dev, check_grads, LOGP_ATOL, REL

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


def _prune_both(fr, ro, V, n, tau, keep, max_len=None):
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, ngram_n=n, tau_num=tau[0], tau_den=tau[1],
                               keep_ratio=keep)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    ml = int(ro.lengths.max()) if max_len is None else max_len
    print(f"[edge] prune N={ro.N} Q={len(ro.group_off) - 1} V={V} n={n} tau={tau} "
          f"keep={keep} max_len={ml}", flush=True)
    out = fr.prune(to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV),
                   to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV), to_dev(ref["class_id"], DEV),
                   to_dev(ref["group_valid"], DEV), V=V,
                   max_group=int(np.diff(ro.group_off).max()), max_len=max(ml, 1),
                   ngram_n=n, tau=tau, keep_ratio=keep, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    assert np.array_equal(out["keep_mask"].cpu().numpy(), ref["keep_mask"])
    assert np.array_equal(out["mdap_count"].cpu().numpy(), ref["mdap_count"])
    nk, tk = out["counts"].cpu().tolist()
    assert nk == len(ref["kept_traj"]) and tk == len(ref["tok_src"])
    assert np.array_equal(out["kept_traj"][:nk].cpu().numpy(), ref["kept_traj"])
    assert np.array_equal(out["kept_tok_off"][:nk + 1].cpu().numpy(), ref["kept_tok_off"])
    assert np.array_equal(out["tok_src"][:tk].cpu().numpy(), ref["tok_src"])
    return ref


@pytest.mark.parametrize("G", [65, 128, 256])
@pytest.mark.parametrize("n", [1, 3])
@pytest.mark.parametrize("keep", [0.0, 0.5])
def test_large_groups(fr, G, n, keep):
    ro = make_rollouts(CONFIGS[3], Q=3, len_range=(1, 30), G=(G,), V=30, seed=500 + G)
    plant_duplicates(ro, p_copy=0.5, p_mutate=0.2, seed=G + n)
    ref = _prune_both(fr, ro, 30, n, (4, 5), keep)
    if keep == 0.0:
        assert ref["keep_mask"].sum() < ro.N  # the duplicates were pruned


def _with_lengths(ro, lengths, V, seed):
    """The same questions and rewards with other trajectory lengths (fresh token ids and
    old / ref noise of the new total)."""
    lengths = np.asarray(lengths, dtype=np.int64)
    off = np.zeros(len(lengths) + 1, dtype=np.int64)
    off[1:] = np.cumsum(lengths)
    T = int(off[-1])
    rng = np.random.default_rng(seed)
    return Rollouts(ro.cfg, ro.group_off, off, lengths, ro.rewards,
                    rng.integers(0, V, size=T).astype(np.int32),
                    rng.normal(0, 0.05, size=T), rng.normal(0, 0.05, size=T),
                    extra={"V": V, "seed": seed})


@pytest.mark.parametrize("n", [1, 2, 3])
def test_max_len_trajectory(fr, n):
    """Trajectories of exactly max_len = 16384 tokens next to short and empty ones."""
    base = make_rollouts(CONFIGS[3], Q=2, len_range=(1, 100), G=(8,), V=60, seed=77)
    L = base.lengths.copy()
    L[0], L[3], L[9], L[5] = 16384, 16384, 12000, 0
    ro = _with_lengths(base, L, 60, seed=78 + n)
    # a near-copy of the long trajectory inside the same question
    ro.token_ids[ro.traj_tok_off[3]:ro.traj_tok_off[4]] = ro.token_ids[0:16384]
    ro.token_ids[ro.traj_tok_off[3] + 5000:ro.traj_tok_off[3] + 5100] = 7
    for keep in (0.0, 0.5):
        _prune_both(fr, ro, 60, n, (4, 5), keep, max_len=16384)


@pytest.mark.parametrize("keep", [0.0, 0.5])
def test_trigrams_at_largest_vocabulary(fr, keep):
    V = (1 << 21) - 1
    ro = make_rollouts(CONFIGS[5], Q=6, len_range=(0, 50), V=V, seed=2121)
    # ids at the top of the range (all 21 bits used) with planted near-copies
    ro.token_ids[:] = V - 1 - (ro.token_ids % 40)
    plant_duplicates(ro, p_copy=0.6, p_mutate=0.1, seed=3)
    ro.token_ids[ro.token_ids < V - 40] = V - 1  # re-drawn positions back to the top ids
    assert ro.token_ids.max() == V - 1
    _prune_both(fr, ro, V, 3, (4, 5), keep)


@pytest.mark.parametrize("case", ["grpo_kl", "gspo", "dapo"])
def test_zero_length_trajectories(fr, case):
    """Many empty trajectories: pruning bit-exact, and the kept (partly empty) sequences
    through the loss and both gradients."""
    # seeds whose draw has >= 3 empty trajectories, >= 2 of them kept
    c, seed = {"grpo_kl": (3, 951), "gspo": (5, 928), "dapo": (4, 907)}[case]
    pb = Problem(c, DEV, Q=6, len_range=(0, 40), V=700, d=64, seed=seed)
    L = pb.ro.lengths
    assert (L == 0).sum() >= 3
    koff = pb.pr["kept_tok_off"]
    assert (np.diff(koff) == 0).sum() >= 2, "no empty kept sequence in this draw"
    ref = pb.oracle_loss()
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    out = pb.run_gpu(fr, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    assert np.array_equal(out["prune"]["keep_mask"].cpu().numpy(), pb.pr["keep_mask"])
    call = out["call"]
    T = out["t_kept"]
    assert T == len(pb.src)
    assert np.abs(call.logp[:T].double().cpu().numpy() - pb.logp_exact).max() < LOGP_ATOL
    assert abs(call.loss.item() - ref["loss"]) <= REL * max(abs(ref["loss"]), 1e-12)
    assert int(call.stats[0].item()) == ref["clipped"]
    check_grads(pb.H64[pb.src], pb.W64, pb.y, ref["g"], call.dhidden[:T].double().cpu().numpy(),
                call.dW.double().cpu().numpy(), ref["dH"], ref["dW"],
                dg=ref["dg"], lse=pb.lse_exact)


@pytest.mark.parametrize("accumulate", [False, True])
def test_all_kept_sequences_empty(fr, accumulate):
    """S > 0 kept sequences, all of length 0 (T = 0), with a NaN-filled workspace: the loss
    is 0, dW is exactly zero (or left as it was when accumulating), nothing reads the
    workspace's stale contents."""
    d, V, S = 64, 300, 3
    H = torch.randn(4, d).bfloat16().to(DEV)
    W = (0.02 * torch.randn(V, d)).bfloat16().to(DEV)
    off = torch.zeros(S + 1, dtype=torch.int64)
    dW0 = torch.full((V, d), 0.25, dtype=torch.float32, device=DEV)
    dW = dW0.clone() if accumulate else torch.full((V, d), float("nan"), device=DEV)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    call = fr.LossCall(H, W, torch.zeros(4, dtype=torch.int32, device=DEV),
                       torch.zeros(4, device=DEV), off.to(DEV), off,
                       torch.ones(S, device=DEV), need_dhidden=True, dW=dW,
                       dW_accumulate=accumulate, status=st, T=0)
    call.ws.fill_(255)  # every float / bfloat16 in it reads as NaN
    call.loss.fill_(float("nan"))
    call.run()
    torch.cuda.synchronize()
    assert st.item() == 0
    assert call.loss.item() == 0.0
    if accumulate:
        assert torch.equal(call.dW, dW0)
    else:
        assert torch.count_nonzero(call.dW).item() == 0
    assert call.stats[0].item() == 0.0
