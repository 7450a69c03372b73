"""Benchmark of one FastRL GRPO hot-path step on one MI355X.

A step is the whole hot path over one batch of seeded synthetic rollouts shaped like
the Qwen2.5-VL-7B GRPO setting (64 prompts x G=8 rollouts, response lengths
U[128, 1024], d = 3584, V = 152064, bf16 hidden/W, KL to a reference at beta = 0.04,
clip 0.2, keep ratio 0.5):

  fastrl_advantage -> fastrl_prune (MDAP + budget + compaction) -> read the kept counts
  -> fastrl_policy_loss_fwd_bwd on the kept tokens (logits GEMM with online log-sum-exp,
  loss, dhidden and dW GEMMs).

Inputs are resident in HBM before timing.  The reported value is kept tokens per second
of the whole step.  ``roofline`` describes the dominant kernel, timed with HIP events on
its launch stream during the timed steps; ``cpu_baseline`` times the fp64 oracle on a
bounded sample of the same workload.  ``rows`` (after the timed steps, skipped with
--no-rows) times the parts beyond the step on the same workload: pruning with
continuous-reward groups, the DP-alignment fill, the entropy accumulator (one loss call with
and without it), the forward-only log-prob pass of the old and ref policies, and the AdamW
update of W (bytes per second against HBM).  Every call of the warmup and timed steps
reports into one device status word; any bit other than the informational SHIFT_REDO makes
the run exit with status 3 and no result line.

usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 3] [--no-cpu]
                       [--no-rows]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X dense fp32 MFMA
SHIFT_REDO = 0x40           # informational status bit (rows re-evaluated with a shift)
DEFAULT_SLAB = 32768        # the library's slab when slab_tokens is 0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=3)
    ap.add_argument("--slab", type=int, default=0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=3072)
    ap.add_argument("--cpu-tokens-1t", type=int, default=16,
                    help="tokens of the one-thread oracle sample (0: skip it)")
    ap.add_argument("--no-rows", action="store_true",
                    help="skip the timings of the additional rows")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run one plain device-to-device copy of this many MiB (a "
                         "known-size reference for the HBM byte counters)")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "lmhead_qwen2.5-vl-7b_grpo_hbm_traffic.md")
KERNEL_SRC = os.path.join(ROOT, "paper_2609_36932_amd", "csrc", "lmhead.hip")


def kernel_source_hash():
    import hashlib
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary, or None when
    there is none or the kernel source changed since the counters were taken."""
    try:
        for line in open(TRAFFIC_FILE):
            if line.startswith("TRAFFIC_JSON "):
                rec = json.loads(line[len("TRAFFIC_JSON "):])
                if rec.get("source_hash") != kernel_source_hash():
                    return None
                k = rec.get("kernels", {}).get(kernel)
                return None if k is None else k["bytes_per_launch"]
    except OSError:
        return None
    return None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def make_inputs(cfg, dev, fr):
    import torch
    from synth import make_rollouts, make_dense
    ro = make_rollouts(cfg)
    H, W = make_dense(cfg, ro.T_total, device=dev)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    inp = dict(rewards=t(ro.rewards), group_off=t(ro.group_off), token_ids=t(ro.token_ids),
               traj_tok_off=t(ro.traj_tok_off), H=H, W=W)
    # old / ref log-probs = current log-probs + N(0, 0.05): evaluate the current policy's
    # log-probs of the kept tokens once, untimed, with the library itself
    adv, cls, valid = fr.advantage(inp["rewards"], inp["group_off"],
                                   drop_uniform=cfg.drop_uniform)
    pr = fr.prune(inp["token_ids"], inp["traj_tok_off"], inp["rewards"], inp["group_off"],
                  cls, valid, V=cfg.V, max_group=int(np.diff(ro.group_off).max()),
                  max_len=int(ro.lengths.max()), keep_ratio=cfg.keep_ratio)
    tk = int(pr["counts"][1].item())
    src = pr["tok_src"][:tk]
    lp, _ = fr.token_logprob(H, W, inp["token_ids"], row_index=src)
    old = torch.full((ro.T_total,), float("nan"), device=dev)
    ref = torch.full((ro.T_total,), float("nan"), device=dev)
    srcl = src.long()
    old[srcl] = lp + t(ro.old_noise)[srcl].float()
    ref[srcl] = lp + t(ro.ref_noise)[srcl].float()
    inp.update(old=old, ref=ref if cfg.beta else None)
    torch.cuda.synchronize()
    return ro, inp


def cpu_baseline(cfg, ro, inp, n_tokens, n_tokens_1t=0):
    """The oracle, as it stands, on a bounded sample: advantage + pruning + compaction of
    the whole batch, then the LM-head forward, loss and full backward (dH and dW at full
    V x d) for the first kept sequences holding >= n_tokens tokens."""
    import oracle
    blas = "unknown"
    try:
        from threadpoolctl import threadpool_info
        info = threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] + [1])
        blas = ",".join(sorted({i.get("internal_api", "?") for i in info if i.get("user_api") == "blas"})) or blas
    except Exception:
        cores = os.cpu_count()
    cpu = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    H = inp["H"]
    Wd = inp["W"].float().cpu().numpy().astype(np.float64)
    old = inp["old"].cpu().numpy()
    ref = inp["ref"].cpu().numpy() if inp["ref"] is not None else None

    def run(tokens, cut=False):
        """Whole kept sequences holding >= tokens tokens; with cut, exactly the first
        tokens kept tokens (the last sequence truncated)."""
        t0 = time.perf_counter()
        pr = oracle.hot_path_step(ro.rewards, ro.group_off, ro.token_ids, ro.traj_tok_off,
                                  lmhead=False, keep_ratio=cfg.keep_ratio,
                                  drop_uniform=cfg.drop_uniform)
        koff = pr["kept_tok_off"]
        S = int(np.searchsorted(koff, tokens)) if koff[-1] >= tokens else len(koff) - 1
        S = max(1, min(S, len(koff) - 1))
        if cut:
            koff = np.minimum(koff, tokens)
        src = pr["tok_src"][:koff[S]]
        Hk = H[torch_index(src, H.device)].float().cpu().numpy().astype(np.float64)
        y = ro.token_ids[src].astype(np.int64)
        logp, lse = oracle.token_logprob(Hk, Wd, y)
        loss, g, _ = oracle.policy_loss(logp, old[src].astype(np.float64),
                                        None if ref is None else ref[src].astype(np.float64),
                                        koff[:S + 1], pr["adv"][pr["kept_traj"][:S]],
                                        algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low,
                                        eps_high=cfg.eps_high, beta=cfg.beta)
        oracle.lmhead_backward(Hk, Wd, y, lse, g)
        return S, len(src), time.perf_counter() - t0

    S, n, dt = run(n_tokens)
    res = dict(value=n / dt, unit="kept tokens/s", cores=int(cores), kind="oracle",
               cpu=cpu, blas=blas,
               sample=f"whole batch advantage+MDAP+compaction, then LM-head fwd + loss + "
                      f"full bwd (dH, dW at V={cfg.V}, d={cfg.d}) in fp64 for the first "
                      f"{S} kept sequences ({n} tokens); {dt:.1f} s")
    if n_tokens_1t > 0:
        try:
            from threadpoolctl import threadpool_limits
            with threadpool_limits(limits=1):
                S1, n1, dt1 = run(n_tokens_1t, cut=True)
            res["one_thread"] = dict(value=n1 / dt1, unit="kept tokens/s", cores=1,
                                     sample=f"the same for the first {n1} kept tokens "
                                            f"({S1} sequences, the last one cut) with one "
                                            f"BLAS thread; {dt1:.1f} s")
        except ImportError:
            res["one_thread"] = None
    return res


def _time_gpu(fn, reps):
    """Average ms of fn() over reps calls on the current stream (HIP events)."""
    import torch
    fn()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        fn()
    b.record()
    b.synchronize()
    return a.elapsed_time(b) / reps


def extra_rows(cfg, ro, inp, fr, max_group, max_len, last, args):
    """Timings of the rows beyond the hot path, on the same workload: pruning with
    continuous-reward groups, the entropy accumulator, the AdamW step on W, the DP fill."""
    import torch
    import oracle
    from synth import continuous_rewards
    dev = inp["H"].device
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    rows = {}
    # the step's small stages on the workload's own rewards: advantage (A1), and pruning with
    # the compaction of the kept tokens (A2 + A3); algorithmic bytes: A1 reads the rewards and
    # group offsets and writes advantage, class and validity; A2 + A3 read every token id once,
    # write and read back one 8-byte n-gram key per token, and write the kept-token index
    N, Q, Tt = len(ro.rewards), len(ro.group_off) - 1, int(ro.T_total)
    a_ms = _time_gpu(lambda: fr.advantage(inp["rewards"], inp["group_off"],
                                          drop_uniform=cfg.drop_uniform), 50)
    adv0, cls0, valid0 = fr.advantage(inp["rewards"], inp["group_off"],
                                      drop_uniform=cfg.drop_uniform)
    p_ms = _time_gpu(lambda: fr.prune(inp["token_ids"], inp["traj_tok_off"], inp["rewards"],
                                      inp["group_off"], cls0, valid0, V=cfg.V,
                                      max_group=max_group, max_len=max_len,
                                      keep_ratio=cfg.keep_ratio), 20)
    a_bytes = 4 * N + 4 * (Q + 1) + 4 * N + 4 * N + Q
    p_bytes = 4 * Tt + 16 * Tt + 4 * last["t_kept"] + 8 * (N + 1)
    rows["small_stages"] = dict(
        advantage_us=a_ms * 1e3, advantage_bytes=a_bytes,
        advantage_GBps=a_bytes / (a_ms * 1e-3) / 1e9,
        prune_compact_us=p_ms * 1e3, prune_compact_bytes=p_bytes,
        prune_compact_GBps=p_bytes / (p_ms * 1e-3) / 1e9, hbm_peak_GBps=8000.0,
        note="latency-bound: a few launches over KB to a few MB (the loss kernel is timed "
             "inside the loss call; see the kernel trace)")
    # N1: continuous groups |A_i - A_j| < 1e-4 (continuous rewards of the same batch shape)
    rw = continuous_rewards(ro.group_off, seed=cfg.seed)
    rw_d = t(rw)
    adv, cls, valid = fr.advantage(rw_d, inp["group_off"])
    kw = dict(V=cfg.V, max_group=max_group, max_len=max_len, keep_ratio=cfg.keep_ratio)
    plain = _time_gpu(lambda: fr.prune(inp["token_ids"], inp["traj_tok_off"], rw_d,
                                       inp["group_off"], cls, valid, **kw), 20)
    cont = _time_gpu(lambda: fr.prune(inp["token_ids"], inp["traj_tok_off"], rw_d,
                                      inp["group_off"], cls, valid, adv=adv, group_eps=1e-4,
                                      **kw), 20)
    t0 = time.perf_counter()
    oracle.hot_path_step(rw, ro.group_off, ro.token_ids, ro.traj_tok_off, lmhead=False,
                         keep_ratio=cfg.keep_ratio, group_eps=1e-4)
    rows["continuous_groups_prune"] = dict(
        ms=cont, ms_bit_equal_classes=plain, oracle_s=time.perf_counter() - t0,
        note="fastrl_prune_ex, eps 1e-4, whole batch incl. compaction; latency-bound")
    # N4: DP fill to a multiple of 8 ranks
    fill = _time_gpu(lambda: fr.prune(inp["token_ids"], inp["traj_tok_off"], rw_d,
                                      inp["group_off"], cls, valid, adv=adv, dp_align=8,
                                      **kw), 20)
    rows["dp_align_fill_prune"] = dict(ms=fill, ms_without=plain, d=8)
    # N2: entropy fused into the log-sum-exp pass: one loss call of the timed step with and
    # without the extra accumulator
    call = last["call"]
    koff = last["kept_tok_off_host"]
    pr = last["prune"]
    mk = lambda ent: fr.LossCall(inp["H"], inp["W"], inp["token_ids"], inp["old"],
                                 pr["kept_tok_off"], koff, last["adv"], ref_logp=inp["ref"],
                                 seq_index=pr["kept_traj"], row_index=pr["tok_src"],
                                 algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low,
                                 eps_high=cfg.eps_high, beta=cfg.beta, T=last["t_kept"],
                                 need_entropy=ent, slab_tokens=args.slab)
    del call
    c0 = mk(False)
    base_ms = _time_gpu(c0.run, 1)
    del c0
    torch.cuda.empty_cache()
    c1 = mk(True)
    ent_ms = _time_gpu(c1.run, 1)
    mean_ent = float(c1.entropy_sum.item()) / max(last["t_kept"], 1)
    del c1
    torch.cuda.empty_cache()
    rows["entropy_in_lse_pass"] = dict(ms_loss_call=ent_ms, ms_loss_call_without=base_ms,
                                       overhead=ent_ms / base_ms - 1.0,
                                       mean_entropy=mean_ent)
    # the old and ref passes of the step (Table timing_breakdown's timing_old / timing_ref):
    # forward-only log-probs of the kept tokens, no exp-logit slab
    tk = last["t_kept"]
    src = pr["tok_src"]
    st = torch.zeros(1, dtype=torch.int32, device=dev)
    lp_ms = _time_gpu(lambda: fr.token_logprob(inp["H"], inp["W"], inp["token_ids"],
                                               row_index=src, T=tk, status=st), 5)
    assert int(st.item()) == 0, fr.status_names(int(st.item()))
    lp_tf = 2.0 * cfg.V * cfg.d * tk / (lp_ms * 1e-3) / 1e12
    rows["token_logprob_old_ref_pass"] = dict(
        ms=lp_ms, kept_tokens=tk, kept_tokens_per_s=tk / (lp_ms * 1e-3), tflops=lp_tf,
        frac_of_peak=lp_tf / PEAK_BF16_TFLOPS,
        note="fastrl_token_logprob over the kept tokens (2 V d FLOP per token)")
    # N3: AdamW on W (float32 master, moments, dW; bf16 copy): 30 bytes per parameter
    n = cfg.V * cfg.d
    th = inp["W"].float().reshape(-1).contiguous()
    g = torch.empty_like(th).normal_(0, 1e-3)
    m, v = torch.zeros_like(th), torch.zeros_like(th)
    wb = torch.empty(n, dtype=torch.bfloat16, device=dev)
    ms = _time_gpu(lambda: fr.adamw_step(th, g, m, v, step=1, w_bf16=wb), 10)
    gbs = 30.0 * n / (ms * 1e-3) / 1e9
    sample = 1 << 22
    th_h, g_h = th[:sample].double().cpu().numpy(), g[:sample].double().cpu().numpy()
    t0 = time.perf_counter()
    oracle.adamw_step(th_h, g_h, np.zeros(sample), np.zeros(sample), 1)
    o_s = time.perf_counter() - t0
    rows["adamw_W"] = dict(ms=ms, params=n, bytes_per_param=30, achieved_GBps=gbs,
                           hbm_peak_GBps=8000.0, frac=gbs / 8000.0,
                           oracle_params_per_s=sample / o_s)
    del th, g, m, v, wb
    torch.cuda.empty_cache()
    return rows


def torch_index(src, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(src)).long().to(dev)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path is "
              "built for one MI355X and multi-GPU sharding is a design note, not a run.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2609_36932_amd as fr
    from synth import CONFIGS
    cfg = CONFIGS[args.workload]
    dev = torch.device("cuda:0")
    log(f"[bench] workload {cfg.name}: generating inputs")
    ro, inp = make_inputs(cfg, dev, fr)
    max_group = int(np.diff(ro.group_off).max())
    max_len = int(ro.lengths.max())

    # device status word of every call in the warmup and timed steps: read once after the
    # timed loop; a data fault or a timed-out stage hand-over invalidates the line
    status = torch.zeros(1, dtype=torch.int32, device=dev)

    def step():
        return fr.hot_path_step(
            inp["rewards"], inp["group_off"], inp["token_ids"], inp["traj_tok_off"],
            inp["H"], inp["W"], inp["old"], inp["ref"], V=cfg.V, max_group=max_group,
            max_len=max_len, algo=cfg.algo, norm=cfg.norm, eps_low=cfg.eps_low,
            eps_high=cfg.eps_high, beta=cfg.beta, ngram_n=cfg.ngram_n,
            tau=(cfg.tau_num, cfg.tau_den), keep_ratio=cfg.keep_ratio,
            drop_uniform=cfg.drop_uniform, slab_tokens=args.slab, status=status)

    for i in range(args.warmup):
        out = step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {i + 1}/{args.warmup} done")
    if args.copy_probe_mib:
        n = args.copy_probe_mib << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b
        log(f"[bench] copy probe of {args.copy_probe_mib} MiB done")
    fr.profile_reset()
    fr.profile_enable(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    kept = 0
    for i in range(args.steps):
        out = step()
        kept += out["t_kept"]
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    fr.profile_enable(False)
    log(f"[bench] {args.steps} timed steps in {elapsed:.3f} s")
    word = int(status.item())
    fatal = word & ~SHIFT_REDO
    if fatal:
        log(f"[bench] INVALID: device status {word:#x} {fr.status_names(word)} after the "
            "warmup and timed steps; no result line")
        sys.exit(3)
    slab_begin, slab_max = out["call"].slab_plan()
    kinds = {fr.K_LOGITS_FWD: "logits_fwd", fr.K_DHIDDEN: "dhidden", fr.K_DW: "dW",
             fr.K_BACKWARD: "backward"}
    per = {}
    for k, name in kinds.items():
        ms, n, fl = fr.profile_read(k)
        if n:
            per[name] = dict(ms_total=ms, launches=n, tflops=fl / (ms * 1e-3) / 1e12,
                             avg_ms=ms / n, flops_per_launch=fl / n)
    dom = max(per, key=lambda k: per[k]["ms_total"])
    peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    ach = per[dom]["tflops"]
    t_kept = out["t_kept"]
    gemm_ms = sum(v["ms_total"] for v in per.values()) / args.steps
    useful = 6.0 * cfg.V * cfg.d * t_kept / (elapsed / args.steps) / 1e12
    res = {
        "metric": "kept tokens/s for log-prob+loss fwd/bwd at 7B LM-head shape; % bf16 MFMA peak",
        "value": kept / elapsed,
        "unit": "kept tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * elapsed / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded rollouts; random-init bf16 hidden states and LM-head weights)",
        "config": {"workload": f"{cfg.name}: {cfg.Q} prompts x G={cfg.G[0]}, lengths "
                               f"U[{cfg.len_lo},{cfg.len_hi}], d={cfg.d}, V={cfg.V}, "
                               f"keep ratio {cfg.keep_ratio}, beta {cfg.beta}",
                   "kept_tokens_per_step": t_kept, "kept_sequences": out["n_kept"],
                   "total_tokens": ro.T_total, "parallelism": "single GPU",
                   "slab_tokens": args.slab or DEFAULT_SLAB, "slabs": len(slab_begin) - 1,
                   "max_slab_tokens": slab_max},
        "status_word": word,
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": ach, "peak": peak,
                     "unit": "TFLOP/s", "frac": ach / peak,
                     "traffic": measured_traffic(dom) if cfg.name == CONFIGS[3].name else None},
        "useful_frac_of_step": useful / peak,
        "kernels": per,
        "gemm_ms_per_step": gemm_ms,
    }
    if not args.no_rows:
        log("[bench] timing the additional rows (continuous groups, entropy, AdamW, DP fill)")
        res["rows"] = extra_rows(cfg, ro, inp, fr, max_group, max_len, out, args)
    if not args.no_cpu:
        log("[bench] timing the oracle on a CPU sample")
        res["cpu_baseline"] = cpu_baseline(cfg, ro, inp, args.cpu_tokens, args.cpu_tokens_1t)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
