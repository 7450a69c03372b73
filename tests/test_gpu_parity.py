"""GPU parity of the HIP path (called through the C ABI) against the fp64 oracle on the
same seeded inputs, at sizes the oracle finishes in seconds that still span several
256-wide tiles with ragged tails.  Bars: masks / indices / offsets bit-exact; log-probs
2e-3 absolute; loss and gradients 1e-2 relative (also for the softmax part of the
gradients alone)."""
import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, make_rollouts
from tests._parity import (Problem, to_dev, rel_fro, check_grads, LOGP_ATOL, REL)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_36932_amd as m
    return m


DEV = "cuda:0"


def _status():
    return torch.zeros(1, dtype=torch.int32, device=DEV)


@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
def test_advantage(fr, c):
    ro = make_rollouts(CONFIGS[c])
    cfg = CONFIGS[c]
    adv, cls, valid = oracle.group_advantage(ro.rewards, ro.group_off,
                                             drop_uniform=cfg.drop_uniform)
    st = _status()
    a, k, v = fr.advantage(to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV),
                           drop_uniform=cfg.drop_uniform, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    np.testing.assert_allclose(a.cpu().numpy(), adv, rtol=1e-6, atol=1e-6)
    assert np.array_equal(k.cpu().numpy(), cls)
    assert np.array_equal(v.cpu().numpy(), valid)


def _prune_gpu(fr, ro, cls, valid, V, n, tau, keep):
    st = _status()
    out = fr.prune(to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV),
                   to_dev(ro.rewards, DEV), to_dev(ro.group_off, DEV), to_dev(cls, DEV),
                   to_dev(valid, DEV), V=V, max_group=int(np.diff(ro.group_off).max()),
                   max_len=int(ro.lengths.max()), ngram_n=n, tau=tau, keep_ratio=keep,
                   status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    return out


def _check_prune(out, ref, N):
    assert np.array_equal(out["keep_mask"].cpu().numpy(), ref["keep_mask"])
    assert np.array_equal(out["mdap_count"].cpu().numpy(), ref["mdap_count"])
    nk, tk = out["counts"].cpu().tolist()
    assert nk == len(ref["kept_traj"]) and tk == len(ref["tok_src"])
    assert np.array_equal(out["kept_traj"][:nk].cpu().numpy(), ref["kept_traj"])
    assert np.array_equal(out["kept_tok_off"][:nk + 1].cpu().numpy(), ref["kept_tok_off"])
    assert np.array_equal(out["tok_src"][:tk].cpu().numpy(), ref["tok_src"])


@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
def test_prune_full_config(fr, c):
    """Pruning, budget and compaction at each workload's full size: bit-exact."""
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=cfg.keep_ratio,
                               drop_uniform=cfg.drop_uniform)
    out = _prune_gpu(fr, ro, ref["class_id"], ref["group_valid"], cfg.V, 1, (4, 5),
                     cfg.keep_ratio)
    _check_prune(out, ref, ro.N)


@pytest.mark.parametrize("n", [1, 2, 3])
@pytest.mark.parametrize("tau", [(4, 5), (0, 1), (2, 1), (1, 1), (1, 2)])
@pytest.mark.parametrize("keep", [0.0, 0.5])
def test_prune_planted_duplicates(fr, n, tau, keep):
    """Near-duplicate rollouts inside each question so the Jaccard test actually prunes."""
    from synth import plant_duplicates
    cfg = CONFIGS[5]
    ro = make_rollouts(cfg, Q=24, len_range=(1, 40), V=40, seed=123 + n)
    plant_duplicates(ro, p_copy=0.7, p_mutate=0.2, seed=n)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, ngram_n=n, tau_num=tau[0], tau_den=tau[1],
                               keep_ratio=keep)
    out = _prune_gpu(fr, ro, ref["class_id"], ref["group_valid"], 40, n, tau, keep)
    _check_prune(out, ref, ro.N)
    if tau == (4, 5) and keep == 0.0:
        assert ref["keep_mask"].sum() < ro.N  # the planted duplicates were pruned


def test_prune_bad_token_flags_status(fr):
    cfg = CONFIGS[1]
    ro = make_rollouts(cfg)
    ro.token_ids[5] = cfg.V + 3
    ref = oracle.group_advantage(ro.rewards, ro.group_off)
    st = _status()
    fr.prune(to_dev(ro.token_ids, DEV), to_dev(ro.traj_tok_off, DEV), to_dev(ro.rewards, DEV),
             to_dev(ro.group_off, DEV), to_dev(ref[1], DEV), to_dev(ref[2], DEV), V=cfg.V,
             max_group=8, max_len=64, keep_ratio=0.5, status=st)
    torch.cuda.synchronize()
    assert st.item() & 0x2


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("V,d", [(1000, 64), (4096, 256), (777, 136)])
def test_token_logprob(fr, dtype, V, d):
    rng = np.random.default_rng(V + d)
    T = 613
    H = rng.normal(size=(T, d)).astype(np.float32)
    W = (0.05 * rng.normal(size=(V, d))).astype(np.float32)
    if dtype == "bf16":
        Ht, Wt = torch.from_numpy(H).bfloat16(), torch.from_numpy(W).bfloat16()
    else:
        Ht, Wt = torch.from_numpy(H), torch.from_numpy(W)
    y = rng.integers(0, V, size=T).astype(np.int32)
    # a gather through row_index (every other row, reversed)
    rows = np.arange(T)[::-2].astype(np.int32).copy()
    lp_ref, lse_ref = oracle.token_logprob(Ht.double().numpy()[rows], Wt.double().numpy(),
                                           y[rows])
    st = _status()
    lp, lse = fr.token_logprob(Ht.to(DEV), Wt.to(DEV), to_dev(y, DEV), row_index=to_dev(rows, DEV),
                               status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    assert np.abs(lp.cpu().numpy() - lp_ref).max() < LOGP_ATOL
    assert np.abs(lse.cpu().numpy() - lse_ref).max() < LOGP_ATOL


CASES = {
    # cfg id, overrides
    "grpo_kl_bf16": (3, dict(Q=6, len_range=(20, 90), V=1000, d=136)),
    "dapo_bf16": (4, dict(Q=5, len_range=(10, 120), V=1291, d=64)),
    "gspo_bf16": (5, dict(Q=6, len_range=(30, 100), V=900, d=96)),
    "grpo_tokmean_bf16": (2, dict(Q=6, len_range=(5, 70), V=600, d=128)),
    "grpo_f32": (1, dict(Q=4, len_range=(16, 64), V=1500, d=72)),
    "gspo_f32": (5, dict(Q=4, len_range=(8, 60), V=700, d=64, dtype="f32")),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("slab", [0, 150])
def test_hot_path_small(fr, case, slab):
    c, kw = CASES[case]
    pb = Problem(c, DEV, **kw)
    ref = pb.oracle_loss()
    st = _status()
    out = pb.run_gpu(fr, slab_tokens=slab, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    assert np.array_equal(out["prune"]["keep_mask"].cpu().numpy(), pb.pr["keep_mask"])
    call = out["call"]
    T = out["t_kept"]
    assert T == len(pb.src)
    lp = call.logp[:T].double().cpu().numpy()
    assert np.abs(lp - pb.logp_exact).max() < LOGP_ATOL
    assert np.abs(call.lse[:T].double().cpu().numpy() - pb.lse_exact).max() < LOGP_ATOL
    loss = float(call.loss.item())
    scale = max(abs(ref["loss"]), 1e-3 * np.abs(ref["g"]).sum() / max(T, 1))
    assert abs(loss - ref["loss"]) <= REL * max(abs(ref["loss"]), 1e-12), (loss, ref["loss"])
    assert int(call.stats[0].item()) == ref["clipped"]
    Hk = pb.H64[pb.src]
    errs = check_grads(Hk, pb.W64, pb.y, ref["g"], call.dhidden[:T].double().cpu().numpy(),
                       call.dW.double().cpu().numpy(), ref["dH"], ref["dW"],
                       dg=ref["dg"], lse=pb.lse_exact, u=pb.fold_u)
    print(case, slab, errs)


def test_cfg1_full(fr):
    """The tiny fp32 workload end to end at its full size."""
    pb = Problem(1, DEV)
    ref = pb.oracle_loss()
    st = _status()
    out = pb.run_gpu(fr, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0
    call = out["call"]
    T = out["t_kept"]
    assert np.abs(call.logp[:T].double().cpu().numpy() - pb.logp_exact).max() < 1e-4
    assert abs(call.loss.item() - ref["loss"]) <= 1e-4 * abs(ref["loss"])
    check_grads(pb.H64[pb.src], pb.W64, pb.y, ref["g"], call.dhidden[:T].double().cpu().numpy(),
                call.dW.double().cpu().numpy(), ref["dH"], ref["dW"], rel=1e-4, dg=pb.g_dev(1e-6),
                lse=pb.lse_exact, u=pb.fold_u)


def test_large_logits_take_the_shifted_path(fr):
    """Logits far outside exp's float range: rows are re-evaluated with a per-row shift and
    the results still match."""
    pb = Problem(3, DEV, Q=3, len_range=(20, 60), V=700, d=64, h_std=40.0, w_std=0.2)
    ref = pb.oracle_loss()
    st = _status()
    out = pb.run_gpu(fr, status=st)
    torch.cuda.synchronize()
    call = out["call"]
    T = out["t_kept"]
    assert call.stats[1].item() > 0  # some rows needed the shift
    err = np.abs(call.logp[:T].double().cpu().numpy() - pb.logp_exact).max()
    err_lse = np.abs(call.lse[:T].double().cpu().numpy() - pb.lse_exact).max()
    print(f"shifted-path logp max error {err:.3e}, lse {err_lse:.3e}")
    assert err < LOGP_ATOL and err_lse < LOGP_ATOL, (err, err_lse)
    check_grads(pb.H64[pb.src], pb.W64, pb.y, ref["g"], call.dhidden[:T].double().cpu().numpy(),
                call.dW.double().cpu().numpy(), ref["dH"], ref["dW"],
                dg=ref["dg"], lse=pb.lse_exact)


def test_shifted_path_in_some_slabs(fr):
    """Slabs of ~80 tokens where only the rows of every third kept sequence have logits of
    magnitude ~100 (their hidden rows scaled by 32): exactly those slabs re-evaluate their
    marked token blocks (each slab's flag starts cleared; slabs without a marked row skip the
    second evaluation and merge), and every slab matches the oracle."""
    pb = Problem(3, DEV, Q=4, len_range=(20, 60), V=700, d=64, w_std=0.2)
    koff = pb.pr["kept_tok_off"]
    big = np.concatenate([pb.src[koff[i]:koff[i + 1]] for i in range(0, len(koff) - 1, 3)])
    pb.scale_hidden(big, 32.0)
    ref = pb.oracle_loss()
    st = _status()
    out = pb.run_gpu(fr, slab_tokens=80, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    call = out["call"]
    T = out["t_kept"]
    nslab = len(call.slab_plan()[0]) - 1
    n_big = len(big)
    # every scaled row (|max logit| >= 106) is marked, no other row (|max logit| < 8)
    assert nslab >= 4 and int(call.stats[1].item()) == n_big, (nslab, call.stats[1].item(), n_big)
    err = np.abs(call.logp[:T].double().cpu().numpy() - pb.logp_exact).max()
    err_lse = np.abs(call.lse[:T].double().cpu().numpy() - pb.lse_exact).max()
    assert err < LOGP_ATOL and err_lse < LOGP_ATOL, (err, err_lse)
    assert abs(call.loss.item() - ref["loss"]) <= REL * max(abs(ref["loss"]), 1e-12)
    assert int(call.stats[0].item()) == ref["clipped"]
    check_grads(pb.H64[pb.src], pb.W64, pb.y, ref["g"], call.dhidden[:T].double().cpu().numpy(),
                call.dW.double().cpu().numpy(), ref["dH"], ref["dW"],
                dg=ref["dg"], lse=pb.lse_exact)


@pytest.mark.parametrize("slab", [0, 120])
def test_deterministic(fr, slab):
    """Two runs give the same bits: masks and offsets, the loss, dhidden and dW (with several
    slabs, dW accumulated across them in the same order)."""
    pb = Problem(5, DEV, Q=4, len_range=(30, 80), V=800, d=64)
    a = pb.run_gpu(fr, slab_tokens=slab)
    b = pb.run_gpu(fr, slab_tokens=slab)
    torch.cuda.synchronize()
    nk, tk = a["n_kept"], a["t_kept"]
    assert (nk, tk) == (b["n_kept"], b["t_kept"])
    valid = {"keep_mask": None, "kept_traj": nk, "kept_tok_off": nk + 1, "tok_src": tk}
    for k, n in valid.items():  # entries past the counts are undefined by contract
        assert torch.equal(a["prune"][k][:n], b["prune"][k][:n])
    assert torch.equal(a["call"].loss, b["call"].loss)
    assert torch.equal(a["call"].dW, b["call"].dW)
    assert torch.equal(a["call"].dhidden, b["call"].dhidden)


@pytest.mark.parametrize("skew", [0.7, 1.0])
@pytest.mark.parametrize("slab", [0, 1000])
def test_head_heavy_labels(fr, skew, slab):
    """A token distribution where one id fills most positions (1.0: all of them): one dW row
    sums the one-hot terms of thousands of tokens (through the exp-logit operand).  dW matches
    the oracle and is the same bit for bit on a second run."""
    pb = Problem(3, DEV, Q=8, len_range=(60, 200), V=500, d=64, skew=skew)
    ref = pb.oracle_loss()
    st = _status()
    a = pb.run_gpu(fr, slab_tokens=slab, status=st)
    b = pb.run_gpu(fr, slab_tokens=slab)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    T = a["t_kept"]
    assert T == len(pb.src) and int((pb.y == 0).sum()) > 2000
    call = a["call"]
    check_grads(pb.H64[pb.src], pb.W64, pb.y, ref["g"], call.dhidden[:T].double().cpu().numpy(),
                call.dW.double().cpu().numpy(), ref["dH"], ref["dW"],
                dg=ref["dg"], lse=pb.lse_exact)
    assert torch.equal(call.dW, b["call"].dW)


def test_empty_and_single_token(fr):
    # no kept sequence at all: loss 0, dW zero
    d, V = 64, 300
    H = torch.randn(4, d).bfloat16().to(DEV)
    W = (0.02 * torch.randn(V, d)).bfloat16().to(DEV)
    z = torch.zeros(1, dtype=torch.int64)
    call = fr.policy_loss_fwd_bwd(H, W, torch.zeros(4, dtype=torch.int32, device=DEV),
                                  torch.zeros(4, device=DEV), z.to(DEV), z,
                                  torch.zeros(1, device=DEV), need_dhidden=True)
    torch.cuda.synchronize()
    assert call.loss.item() == 0.0 and torch.count_nonzero(call.dW).item() == 0
    # one sequence of one token against the oracle
    y = np.asarray([7], dtype=np.int32)
    Hn = H[:1].double().cpu().numpy()
    Wn = W.double().cpu().numpy()
    lp, lse = oracle.token_logprob(Hn, Wn, y)
    old = (lp - 0.1).astype(np.float32)
    off = np.asarray([0, 1], dtype=np.int64)
    loss, g, _ = oracle.policy_loss(lp, old.astype(np.float64), None, off, [0.7])
    dH, dW = oracle.lmhead_backward(Hn, Wn, y, lse, g)
    call = fr.policy_loss_fwd_bwd(H[:1].contiguous(), W, to_dev(y, DEV), to_dev(old, DEV),
                                  to_dev(off, DEV), torch.from_numpy(off),
                                  torch.tensor([0.7], device=DEV))
    torch.cuda.synchronize()
    assert abs(call.loss.item() - loss) < 1e-2 * abs(loss)
    assert rel_fro(call.dW.double().cpu().numpy(), dW) < REL
    assert rel_fro(call.dhidden[:1].double().cpu().numpy(), dH) < REL


@pytest.mark.parametrize("which", ["dhidden_only", "dW_only"])
def test_single_backward_gemm(fr, which):
    """One backward GEMM alone (its own launch) gives the same gradient as the joint launch."""
    pb = Problem(3, DEV, Q=4, len_range=(20, 90), V=1000, d=136)
    ref = pb.oracle_loss()
    pr = pb.pr
    cfg = pb.cfg
    call = fr.LossCall(
        pb.H_poisoned.to(DEV), pb.W.to(DEV), to_dev(pb.ro.token_ids, DEV), to_dev(pb.old, DEV),
        to_dev(pr["kept_tok_off"], DEV), torch.from_numpy(pr["kept_tok_off"]),
        to_dev(pr["adv"].astype(np.float32), DEV), ref_logp=to_dev(pb.ref, DEV),
        seq_index=to_dev(pr["kept_traj"].astype(np.int32), DEV),
        row_index=to_dev(pb.src.astype(np.int32), DEV), algo=cfg.algo, norm=cfg.norm,
        eps_low=cfg.eps_low, eps_high=cfg.eps_high, beta=cfg.beta,
        need_dhidden=which == "dhidden_only", need_dW=which == "dW_only").run()
    torch.cuda.synchronize()
    T = len(pb.src)
    if which == "dhidden_only":
        assert call.dW is None
        assert rel_fro(call.dhidden[:T].double().cpu().numpy(), ref["dH"]) < REL
    else:
        assert call.dhidden is None
        assert rel_fro(call.dW.double().cpu().numpy(), ref["dW"]) < REL
