"""GPU parity at the workloads' full sizes (the launch configuration bench.py times).

The oracle cannot evaluate every kept token at the 7B shape (up to 7.5e14 fp64 FLOP), so:
* pruning, budget and compaction are compared whole (bit-exact);
* log-probs and dhidden are compared on a seeded sample of kept tokens (GSPO: on whole
  sampled sequences, whose ratio needs every token), each computed exactly by the oracle;
* dW, dhidden and the loss are checked through properties that hold at any size:
  sum_v dW[v] = 0 (relative to the one-hot part), <dW, W> = <dH, H>, and the reported loss
  equals the loss of the reported log-probs;
* a slab of whole kept sequences (about 1K tokens) at full V x d runs through the same entry
  point and is compared element by element, dW and the per-token entropy included;
* the forward-only fastrl_token_logprob (the old / ref passes) runs on all kept tokens and is
  compared on the same sample;
* test_full_k_dw_rows: dW rows of >= 256 vocabulary ids at full K (every kept token in the
  same call, several slabs), exact from the oracle: the old log-probs clip every sequence
  but a few spread over the batch (g = 0 elsewhere), so the oracle needs the log-sum-exp of
  those few only; the zero rows of dhidden must be exactly zero;
* test_dense_multislab: the first >= 8192 kept tokens of the 7B GRPO + KL workload, all with
  a nonzero gradient, cut into 2048-token slabs: every log-prob, the loss, the clip count,
  >= 256 dW rows and 512 dhidden rows against the oracle.
Gradients: relative Frobenius error and largest per-row relative error <= 1e-2.
Old/ref log-probs are "current + N(0, 0.05)": exact oracle log-probs for every token the
oracle checks, a plain-torch fp32 evaluation for the others.
"""
import numpy as np
import pytest
import torch

import oracle
from synth import CONFIGS, make_rollouts, make_dense
from tests._parity import rel_fro, row_rel, onehot_parts, fold_bounds, soft_excess, LOGP_ATOL, REL

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
N_SAMPLE = 96
SLAB_TOKENS = 1024


@pytest.fixture(scope="module")
def fr():
    assert torch.cuda.is_available()
    import paper_2609_36932_amd as m
    return m


def _torch_logp(H, W, rows, y, chunk=4096):
    """Plain-torch fp32 log-probs of kept tokens (input synthesis only)."""
    Wt = W.float().t().contiguous()
    out = torch.empty(len(rows), dtype=torch.float32, device=H.device)
    for a in range(0, len(rows), chunk):
        b = min(len(rows), a + chunk)
        z = H[rows[a:b]].float() @ Wt
        out[a:b] = z.gather(1, y[a:b, None])[:, 0] - torch.logsumexp(z, dim=1)
        del z
    del Wt
    return out


@pytest.mark.parametrize("c", [2, 3, 4, 5])
def test_full_config(fr, c):
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg)
    print(f"[fullsize] cfg {c} {cfg.name}: T_total={ro.T_total}", flush=True)
    H, W = make_dense(cfg, ro.T_total, device=DEV)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=cfg.keep_ratio,
                               drop_uniform=cfg.drop_uniform)
    src = ref["tok_src"]
    koff = ref["kept_tok_off"]
    T = len(src)
    S = len(koff) - 1
    y_all = ro.token_ids[src].astype(np.int64)
    rng = np.random.default_rng(c)
    W64 = W.double().cpu().numpy()

    def exact(idx):
        Hs = H[torch.from_numpy(src[idx]).long().to(DEV)].double().cpu().numpy()
        lp, lse = oracle.token_logprob(Hs, W64, y_all[idx])
        return Hs, lp, lse

    # tokens the oracle checks: a seeded sample, or two whole sequences for GSPO
    if cfg.algo == "gspo":
        # two short sequences with a nonzero gradient: old = exact + noise makes the sequence
        # ratio exp(-mean noise), so the clip decision is known before any log-prob
        L = np.diff(koff)
        A_k = ref["adv"][ref["kept_traj"]]
        sr = np.exp([-ro.old_noise[src[koff[i]:koff[i + 1]]].mean() for i in range(S)])
        live = ((A_k > 0) & (sr <= 1 + cfg.eps_high)) | ((A_k < 0) & (sr >= 1 - cfg.eps_low))
        cand = [i for i in np.argsort(L, kind="stable") if live[i]]
        assert len(cand) >= 2
        sample = np.concatenate([np.arange(koff[i], koff[i + 1]) for i in cand[:2]])
    else:
        sample = np.sort(rng.choice(T, size=N_SAMPLE, replace=False))
    Hs, lp_s, lse_s = exact(sample)

    # old / ref = current + noise; the current log-prob is exact on the checked tokens
    x = _torch_logp(H, W, torch.from_numpy(src).long().to(DEV),
                    torch.from_numpy(y_all).to(DEV)).double().cpu().numpy()
    x[sample] = lp_s
    old = np.full(ro.T_total, np.nan, dtype=np.float32)
    refl = np.full(ro.T_total, np.nan, dtype=np.float32)
    old[src] = (x + ro.old_noise[src]).astype(np.float32)
    refl[src] = (x + ro.ref_noise[src]).astype(np.float32)
    # poison pruned rows: the kernels must never read them
    pruned = np.ones(ro.T_total, dtype=bool)
    pruned[src] = False
    H[torch.from_numpy(pruned).to(DEV)] = float("nan")

    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    out = fr.hot_path_step(t(ro.rewards), t(ro.group_off), t(ro.token_ids), t(ro.traj_tok_off),
                           H, W, t(old), t(refl) if cfg.beta else None, V=cfg.V,
                           max_group=int(np.diff(ro.group_off).max()),
                           max_len=int(ro.lengths.max()), algo=cfg.algo, norm=cfg.norm,
                           eps_low=cfg.eps_low, eps_high=cfg.eps_high, beta=cfg.beta,
                           keep_ratio=cfg.keep_ratio, drop_uniform=cfg.drop_uniform, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    # pruning + compaction: bit-exact
    assert np.array_equal(out["prune"]["keep_mask"].cpu().numpy(), ref["keep_mask"])
    assert (out["n_kept"], out["t_kept"]) == (S, T)
    assert np.array_equal(out["kept_tok_off_host"].numpy(), koff)
    assert np.array_equal(out["prune"]["tok_src"][:T].cpu().numpy(), src)
    call = out["call"]
    logp = call.logp[:T].double().cpu().numpy()
    assert np.all(np.isfinite(logp))
    # sampled log-probs
    err = np.abs(logp[sample] - lp_s).max()
    assert err < LOGP_ATOL, err
    # g on the checked tokens from oracle-only inputs; their dhidden rows exactly
    A = ref["adv"][ref["kept_traj"]]
    loss_x, g_x, _ = oracle.policy_loss(x, old[src].astype(np.float64),
                                        refl[src].astype(np.float64) if cfg.beta else None,
                                        koff, A, algo=cfg.algo, norm=cfg.norm,
                                        eps_low=cfg.eps_low, eps_high=cfg.eps_high,
                                        beta=cfg.beta)
    g_s = g_x[sample]
    dH_s, _ = oracle.lmhead_backward(Hs, W64, y_all[sample], lse_s, g_s, need_dW=False)
    dH_gpu = call.dhidden[torch.from_numpy(sample).long().to(DEV)].double().cpu().numpy()
    e1 = rel_fro(dH_gpu, dH_s)
    dH1, _ = onehot_parts(Hs, W64, y_all[sample], g_s)
    e2 = soft_excess(dH_gpu, dH_s, dH1, fold_bounds(Hs, W64, y_all[sample], g_s)[0])
    e3 = row_rel(dH_gpu, dH_s)
    assert np.abs(g_s).max() > 0 and e1 < REL and e2 < REL and e3 < REL, (e1, e2, e3)
    # the forward-only entry point (the old / ref passes) on the same kept tokens, full size
    lp_only, lse_only = fr.token_logprob(H, W, t(ro.token_ids), row_index=t(src.astype(np.int32)),
                                         status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    sd = torch.from_numpy(sample).long().to(DEV)
    e_lp = np.abs(lp_only[sd].double().cpu().numpy() - lp_s).max()
    e_lse = np.abs(lse_only[sd].double().cpu().numpy() - lse_s).max()
    assert e_lp < LOGP_ATOL and e_lse < LOGP_ATOL, (e_lp, e_lse)
    assert torch.isfinite(lp_only).all()
    del lp_only, lse_only
    # the reported loss is the loss of the reported log-probs
    loss_gpu = float(call.loss.item())
    loss_prop, _, _ = oracle.policy_loss(logp, old[src].astype(np.float64),
                                         refl[src].astype(np.float64) if cfg.beta else None,
                                         koff, A, algo=cfg.algo, norm=cfg.norm,
                                         eps_low=cfg.eps_low, eps_high=cfg.eps_high,
                                         beta=cfg.beta)
    assert abs(loss_gpu - loss_prop) <= REL * max(abs(loss_prop), 1e-8), (loss_gpu, loss_prop)
    # dW: the vocabulary sum cancels the one-hot part sum_t g_t H_t; <dW, W> = <dH, H>
    dW = call.dW
    Hk = H[torch.from_numpy(src).long().to(DEV)]
    colsum = dW.double().sum(0)
    onehot = (torch.from_numpy(g_x).to(DEV)[:, None] * Hk.double()).sum(0)
    assert colsum.norm().item() <= 1e-2 * onehot.norm().item(), (colsum.norm().item(),
                                                                 onehot.norm().item())
    a = (dW.double() * W.double()).sum().item()
    b = (call.dhidden[:T].double() * Hk.double()).sum().item()
    assert abs(a - b) <= REL * max(abs(a), abs(b)), (a, b)
    del dW, Hk, call, out
    torch.cuda.empty_cache()
    print(f"[fullsize] cfg {c}: T_kept={T} logp err {err:.2e} dH {e1:.2e}/{e2:.2e} "
          f"loss {loss_gpu:.6g} ({loss_prop:.6g})", flush=True)

    # ---- a slab of whole kept sequences at full V x d, element by element
    S2 = int(np.searchsorted(koff, SLAB_TOKENS))
    S2 = max(1, min(S2, S))
    T2 = int(koff[S2])
    idx = np.arange(T2)
    Hs2, lp2, lse2 = exact(idx)
    old2 = np.full(ro.T_total, np.nan, dtype=np.float32)
    ref2 = np.full(ro.T_total, np.nan, dtype=np.float32)
    old2[src[:T2]] = (lp2 + ro.old_noise[src[:T2]]).astype(np.float32)
    ref2[src[:T2]] = (lp2 + ro.ref_noise[src[:T2]]).astype(np.float32)
    A2 = ref["adv"][ref["kept_traj"][:S2]]
    off2 = koff[:S2 + 1]
    loss2, g2, info2 = oracle.policy_loss(lp2, old2[src[:T2]].astype(np.float64),
                                          ref2[src[:T2]].astype(np.float64) if cfg.beta else None,
                                          off2, A2, algo=cfg.algo, norm=cfg.norm,
                                          eps_low=cfg.eps_low, eps_high=cfg.eps_high,
                                          beta=cfg.beta)
    dH2, dW2 = oracle.lmhead_backward(Hs2, W64, y_all[:T2], lse2, g2)
    adv_dev = t(ref["adv"].astype(np.float32))
    call2 = fr.LossCall(H, W, t(ro.token_ids), t(old2), t(off2), torch.from_numpy(off2), adv_dev,
                        ref_logp=t(ref2) if cfg.beta else None,
                        seq_index=t(ref["kept_traj"][:S2]), row_index=t(src[:T2].astype(np.int32)),
                        algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low, eps_high=cfg.eps_high,
                        beta=cfg.beta, status=st, need_entropy=True).run()
    torch.cuda.synchronize()
    assert st.item() == 0
    lpg = call2.logp[:T2].double().cpu().numpy()
    assert np.abs(lpg - lp2).max() < LOGP_ATOL
    assert abs(call2.loss.item() - loss2) <= REL * max(abs(loss2), 1e-8)
    assert int(call2.stats[0].item()) == info2["clipped_tokens"]
    ent2 = oracle.token_entropy(Hs2, W64)
    assert np.abs(call2.entropy[:T2].double().cpu().numpy() - ent2).max() < 2e-3
    assert abs(call2.entropy_sum.item() - ent2.sum()) <= 1e-4 * ent2.sum()
    dHg = call2.dhidden[:T2].double().cpu().numpy()
    dWg = call2.dW.double().cpu().numpy()
    dH1, dW1 = onehot_parts(Hs2, W64, y_all[:T2], g2)
    bH, bW = fold_bounds(Hs2, W64, y_all[:T2], g2)
    errs = dict(dH=rel_fro(dHg, dH2), dW=rel_fro(dWg, dW2),
                dH_soft=soft_excess(dHg, dH2, dH1, bH), dW_soft=soft_excess(dWg, dW2, dW1, bW),
                dH_row=row_rel(dHg, dH2), dW_row=row_rel(dWg, dW2))
    print(f"[fullsize] cfg {c} slab of {S2} sequences / {T2} tokens: {errs}", flush=True)
    for k, v in errs.items():
        assert v < REL, (k, v)


def _row_ids(y_all, y_live, V, rng, n_top=96, n_live=96, n_rand=96):
    """>= 256 distinct vocabulary ids: the most frequent labels, labels of live tokens and
    random ids (most of them never a label: their rows are the softmax part alone)."""
    ids, cnt = np.unique(y_all, return_counts=True)
    top = ids[np.argsort(-cnt, kind="stable")[:n_top]]
    live = rng.choice(np.unique(y_live), size=min(n_live, len(np.unique(y_live))), replace=False)
    rows = np.unique(np.concatenate([top, live, rng.choice(V, size=n_rand, replace=False)]))
    while len(rows) < 256:
        rows = np.unique(np.concatenate([rows, rng.choice(V, size=256 - len(rows), replace=False)]))
    return rows


@pytest.mark.parametrize("c", [3, 4, 5])
def test_full_k_dw_rows(fr, c):
    """dW rows at full K against the oracle, element by element."""
    cfg = CONFIGS[c]
    ro = make_rollouts(cfg)
    print(f"[fullK] cfg {c} {cfg.name}: T_total={ro.T_total}", flush=True)
    H, W = make_dense(cfg, ro.T_total, device=DEV)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=cfg.keep_ratio,
                               drop_uniform=cfg.drop_uniform)
    src, koff = ref["tok_src"], ref["kept_tok_off"]
    T, S = len(src), len(koff) - 1
    y_all = ro.token_ids[src].astype(np.int64)
    A = ref["adv"][ref["kept_traj"]]
    L = np.diff(koff)
    W64 = W.double().cpu().numpy()
    # live sequences: nonzero advantage, spread over the batch (so over every slab); for GSPO
    # also a sequence ratio inside the clip window with margin
    sr = np.exp([-ro.old_noise[src[koff[i]:koff[i + 1]]].mean() for i in range(S)])
    ok = A != 0
    if cfg.algo == "gspo":
        ok &= ((A > 0) & (sr <= 1 + cfg.eps_high)) | ((A < 0) & (sr >= 1 - cfg.eps_low))
    cand = np.flatnonzero(ok)
    live_seq = cand[np.linspace(0, len(cand) - 1, 5).round().astype(int)]
    live_seq = np.unique(live_seq)
    live_tok = np.concatenate([np.arange(koff[i], koff[i + 1]) for i in live_seq])
    Hl = H[torch.from_numpy(src[live_tok]).long().to(DEV)].double().cpu().numpy()
    lp_l, lse_l = oracle.token_logprob(Hl, W64, y_all[live_tok])
    # current log-probs: exact on live tokens, plain-torch fp32 elsewhere (input synthesis);
    # every other sequence's old log-probs put its ratio 0.5 past the clip edge on the side
    # that zeroes its gradient (A > 0: rho = e^0.5; A < 0: rho = e^-0.5)
    x = _torch_logp(H, W, torch.from_numpy(src).long().to(DEV),
                    torch.from_numpy(y_all).to(DEV)).double().cpu().numpy()
    x[live_tok] = lp_l
    side = np.repeat(np.sign(A), L)
    o_k = x - 0.5 * side
    o_k[live_tok] = x[live_tok] + ro.old_noise[src[live_tok]]
    old = np.full(ro.T_total, np.nan, dtype=np.float32)
    old[src] = o_k.astype(np.float32)
    loss_x, g_x, _ = oracle.policy_loss(x, old[src].astype(np.float64), None, koff, A,
                                        algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low,
                                        eps_high=cfg.eps_high, beta=0.0)
    dead = np.ones(T, dtype=bool)
    dead[live_tok] = False
    assert np.all(g_x[dead] == 0.0) and np.abs(g_x[live_tok]).max() > 0
    pruned = np.ones(ro.T_total, dtype=bool)
    pruned[src] = False
    H[torch.from_numpy(pruned).to(DEV)] = float("nan")
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    out = fr.hot_path_step(t(ro.rewards), t(ro.group_off), t(ro.token_ids), t(ro.traj_tok_off),
                           H, W, t(old), None, V=cfg.V,
                           max_group=int(np.diff(ro.group_off).max()),
                           max_len=int(ro.lengths.max()), algo=cfg.algo, norm=cfg.norm,
                           eps_low=cfg.eps_low, eps_high=cfg.eps_high, beta=0.0,
                           keep_ratio=cfg.keep_ratio, drop_uniform=cfg.drop_uniform, status=st)
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    call = out["call"]
    nslab = len(call.slab_plan()[0]) - 1
    assert out["t_kept"] == T and nslab >= 2
    rng = np.random.default_rng(100 + c)
    rows = _row_ids(y_all, y_all[live_tok], cfg.V, rng)
    dW_ref = oracle.lmhead_dW_rows(Hl, W64, y_all[live_tok], lse_l, g_x[live_tok], rows)
    dW_gpu = call.dW[torch.from_numpy(rows).long().to(DEV)].double().cpu().numpy()
    e_fro, e_row = rel_fro(dW_gpu, dW_ref), row_rel(dW_gpu, dW_ref)
    # dhidden: live rows against the oracle, the zero-gradient rows exactly zero
    ls = rng.choice(len(live_tok), size=min(256, len(live_tok)), replace=False)
    dH_ref, _ = oracle.lmhead_backward(Hl[ls], W64, y_all[live_tok][ls], lse_l[ls],
                                       g_x[live_tok][ls], need_dW=False)
    dH_gpu = call.dhidden[torch.from_numpy(live_tok[ls]).long().to(DEV)].double().cpu().numpy()
    e_dh = row_rel(dH_gpu, dH_ref)
    dead_idx = torch.from_numpy(np.flatnonzero(dead)).long().to(DEV)
    dead_max = call.dhidden[dead_idx].abs().max().item()
    print(f"[fullK] cfg {c}: T_kept={T} slabs={nslab} live={len(live_tok)} rows={len(rows)} "
          f"dW fro {e_fro:.2e} row {e_row:.2e} dH row {e_dh:.2e} dead dH max {dead_max}",
          flush=True)
    assert e_fro < REL and e_row < REL and e_dh < REL, (e_fro, e_row, e_dh)
    assert dead_max == 0.0


def test_dense_multislab(fr):
    """The first >= 8192 kept tokens of the 7B GRPO + KL workload, every one with a nonzero
    gradient, in 2048-token slabs: log-probs, loss, clip count, dW rows, dhidden rows."""
    cfg = CONFIGS[3]
    ro = make_rollouts(cfg)
    H, W = make_dense(cfg, ro.T_total, device=DEV)
    ref = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                               lmhead=False, keep_ratio=cfg.keep_ratio,
                               drop_uniform=cfg.drop_uniform)
    src, koff = ref["tok_src"], ref["kept_tok_off"]
    S2 = int(np.searchsorted(koff, 8192))
    T2 = int(koff[S2])
    assert T2 >= 8192
    src2 = src[:T2]
    y2 = ro.token_ids[src2].astype(np.int64)
    W64 = W.double().cpu().numpy()
    print(f"[dense] {S2} sequences / {T2} tokens: oracle forward", flush=True)
    H2 = H[torch.from_numpy(src2).long().to(DEV)].double().cpu().numpy()
    lp2, lse2 = oracle.token_logprob(H2, W64, y2)
    old2 = np.full(ro.T_total, np.nan, dtype=np.float32)
    ref2 = np.full(ro.T_total, np.nan, dtype=np.float32)
    old2[src2] = (lp2 + ro.old_noise[src2]).astype(np.float32)
    ref2[src2] = (lp2 + ro.ref_noise[src2]).astype(np.float32)
    A2 = ref["adv"][ref["kept_traj"][:S2]]
    off2 = koff[:S2 + 1]
    loss2, g2, info2 = oracle.policy_loss(lp2, old2[src2].astype(np.float64),
                                          ref2[src2].astype(np.float64), off2, A2,
                                          algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low,
                                          eps_high=cfg.eps_high, beta=cfg.beta)
    assert np.all(g2 != 0.0)
    st = torch.zeros(1, dtype=torch.int32, device=DEV)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    call = fr.LossCall(H, W, t(ro.token_ids), t(old2), t(off2), torch.from_numpy(off2),
                       t(ref["adv"].astype(np.float32)), ref_logp=t(ref2),
                       seq_index=t(ref["kept_traj"][:S2]), row_index=t(src2.astype(np.int32)),
                       algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low, eps_high=cfg.eps_high,
                       beta=cfg.beta, status=st, slab_tokens=2048).run()
    torch.cuda.synchronize()
    assert st.item() == 0, fr.status_names(st.item())
    assert len(call.slab_plan()[0]) - 1 >= 4
    e_lp = np.abs(call.logp[:T2].double().cpu().numpy() - lp2).max()
    assert e_lp < LOGP_ATOL, e_lp
    assert abs(call.loss.item() - loss2) <= REL * abs(loss2), (call.loss.item(), loss2)
    assert int(call.stats[0].item()) == info2["clipped_tokens"]
    rng = np.random.default_rng(8192)
    rows = _row_ids(y2, y2, cfg.V, rng)
    dW_ref = oracle.lmhead_dW_rows(H2, W64, y2, lse2, g2, rows)
    dW_gpu = call.dW[torch.from_numpy(rows).long().to(DEV)].double().cpu().numpy()
    ts = np.sort(rng.choice(T2, size=512, replace=False))
    dH_ref, _ = oracle.lmhead_backward(H2[ts], W64, y2[ts], lse2[ts], g2[ts], need_dW=False)
    dH_gpu = call.dhidden[torch.from_numpy(ts).long().to(DEV)].double().cpu().numpy()
    errs = dict(dW=rel_fro(dW_gpu, dW_ref), dW_row=row_rel(dW_gpu, dW_ref),
                dH=rel_fro(dH_gpu, dH_ref), dH_row=row_rel(dH_gpu, dH_ref), logp=e_lp)
    print(f"[dense] {errs}", flush=True)
    for k, v in errs.items():
        assert v < (LOGP_ATOL if k == "logp" else REL), (k, v)
