"""Python binding of libfastrl (the gfx950 hot path of a FastRL GRPO step).

Argument marshalling only: every step of the path runs in the library's HIP kernels.
PyTorch supplies device memory (``data_ptr``) and the current HIP stream.  The entry
points and their semantics are those of ``include/fastrl.h``:

  advantage            Sec. 3.2, Eq. (advantage) and Eq. (grouping)
  prune                Sec. 3.2 / Alg. 1 Phase 2 (MDAP), keep budget, compaction
  token_logprob        Sec. 3.2, post-pruning evaluation (LM head + log-softmax + gather)
  policy_loss_fwd_bwd  Sec. 3.1 (Eq. 1, Eq. grad): loss, dhidden, dW
  ARS                  Sec. 3.3 / Alg. 1 Phase 1 (host controller)

The library must be built (``python -m paper_2609_36932_amd.build`` or
``__graft_entry__.build()``); importing this module raises if it is missing.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# FASTRL_LIB selects another build of the same library (e.g. a debug build)
LIB_PATH = os.environ.get("FASTRL_LIB", os.path.join(_HERE, "libfastrl.so"))

F32, BF16 = 0, 1
GRPO, DAPO, GSPO = 0, 1, 2
NORM_SEQ_MEAN_TOKEN_MEAN, NORM_TOKEN_MEAN = 0, 1
ALGOS = {"grpo": GRPO, "dapo": DAPO, "gspo": GSPO}
NORMS = {"seq_mean_token_mean": NORM_SEQ_MEAN_TOKEN_MEAN, "token_mean": NORM_TOKEN_MEAN}
K_LOGITS_FWD, K_DHIDDEN, K_DW, K_BACKWARD = 0, 1, 2, 3
STATUS_BITS = {0x1: "BAD_OFFSETS", 0x2: "BAD_TOKEN", 0x4: "GROUP_TOO_BIG",
               0x8: "SEQ_TOO_LONG", 0x10: "BAD_REWARD", 0x20: "BAD_INDEX",
               0x40: "SHIFT_REDO", 0x80: "BAD_GRAD", 0x100: "FILL_SHORT", 0x200: "SYNC_TIMEOUT"}

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")

_lib = ctypes.CDLL(LIB_PATH)

_vp, _i32, _i64, _f32, _f64, _sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                     ctypes.c_float, ctypes.c_double, ctypes.c_size_t)


class LossArgs(ctypes.Structure):
    _fields_ = [
        ("hidden", _vp), ("row_index", _vp), ("W", _vp), ("dtype", _i32), ("d", _i32),
        ("V", _i32), ("S", _i32), ("T", _i64), ("token_ids", _vp), ("old_logp", _vp),
        ("ref_logp", _vp), ("seq_off", _vp), ("seq_off_host", _vp), ("adv", _vp),
        ("seq_index", _vp), ("algo", _i32), ("norm", _i32), ("eps_low", _f32),
        ("eps_high", _f32), ("beta", _f32), ("loss", _vp), ("logp", _vp), ("lse", _vp),
        ("dhidden", _vp), ("dhidden_dtype", _i32), ("dW_accumulate", _i32), ("dW", _vp),
        ("stats", _vp), ("slab_tokens", _i64), ("status", _vp), ("ws", _vp),
        ("ws_bytes", _sz), ("entropy", _vp), ("entropy_sum", _vp),
    ]


class PruneArgs(ctypes.Structure):
    _fields_ = [
        ("token_ids", _vp), ("traj_tok_off", _vp), ("T_total", _i64), ("rewards", _vp),
        ("group_off", _vp), ("class_id", _vp), ("group_valid", _vp), ("Q", _i32), ("N", _i32),
        ("max_group", _i32), ("max_len", _i32), ("V", _i32), ("ngram_n", _i32),
        ("tau_num", _i32), ("tau_den", _i32), ("keep_ratio", _f64), ("keep_mask", _vp),
        ("mdap_count", _vp), ("kept_traj", _vp), ("kept_tok_off", _vp), ("tok_src", _vp),
        ("counts", _vp), ("status", _vp), ("ws", _vp), ("ws_bytes", _sz), ("adv", _vp),
        ("group_eps", _f64), ("class_out", _vp), ("dp_align", _i32),
    ]


class ARSState(ctypes.Structure):
    _fields_ = [("G", _i32), ("pad_", _i32), ("total_steps", _i64),
                ("steps_per_epoch", _i64), ("step", _i64), ("G_ref", _f64), ("G_t", _f64),
                ("sum_mean", _f64), ("sum_max", _f64), ("n_buf", _i64)]


_SIGS = {
    "fastrl_last_error": (ctypes.c_char_p, []),
    "fastrl_version": (ctypes.c_int, []),
    "fastrl_advantage": (ctypes.c_int, [_vp, _vp, _i32, _i32, _i32, _f32, _i32, _vp, _vp, _vp,
                                        _vp, _vp]),
    "fastrl_prune_workspace_size": (_sz, [_i32, _i32, _i64, _i32, _i32]),
    "fastrl_prune": (ctypes.c_int, [_vp, _vp, _i64, _vp, _vp, _vp, _vp, _i32, _i32, _i32,
                                    _i32, _i32, _i32, _i32, _i32, _f64, _vp, _vp, _vp, _vp,
                                    _vp, _vp, _vp, _vp, _sz, _vp]),
    "fastrl_prune_args_size": (_sz, []),
    "fastrl_prune_ex": (ctypes.c_int, [ctypes.POINTER(PruneArgs), _vp]),
    "fastrl_token_logprob_workspace_size": (_sz, [_i64, _i32, _i32, _i32]),
    "fastrl_token_logprob": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i64, _i32, _i32, _vp, _vp,
                                            _vp, _vp, _vp, _sz, _vp]),
    "fastrl_token_logprob_noalloc": (ctypes.c_int, [_vp, _vp, _vp, _i32, _i64, _i32, _i32,
                                                    _vp, _vp, _vp, _vp, _vp]),
    "fastrl_token_logprob_noalloc_scratch_bytes": (_sz, []),
    "fastrl_token_logprob_noalloc_max_chunk": (_i64, [_i32]),
    "fastrl_loss_args_size": (_sz, []),
    "fastrl_policy_loss_workspace_size": (_sz, [ctypes.POINTER(LossArgs)]),
    "fastrl_policy_loss_fwd_bwd": (ctypes.c_int, [ctypes.POINTER(LossArgs), _vp]),
    "fastrl_policy_loss_slab_plan": (ctypes.c_int, [ctypes.POINTER(LossArgs), _vp, _i32,
                                                    ctypes.POINTER(_i64)]),
    "fastrl_adamw_step": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _f32, _f32,
                                         _f32, _f32, _f32, _f32, _vp, _vp]),
    "fastrl_ars_init": (ctypes.c_int, [ctypes.POINTER(ARSState), _i32, _i64, _i64]),
    "fastrl_ars_next_n": (ctypes.c_int32, [ctypes.POINTER(ARSState)]),
    "fastrl_ars_observe": (ctypes.c_int, [ctypes.POINTER(ARSState), _vp, _vp, _i32]),
    "fastrl_profile_enable": (ctypes.c_int, [_i32]),
    "fastrl_profile_reset": (ctypes.c_int, []),
    "fastrl_profile_read": (ctypes.c_int, [_i32, ctypes.POINTER(_f64), ctypes.POINTER(_i64),
                                           ctypes.POINTER(_f64)]),
}
for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args

if _lib.fastrl_loss_args_size() != ctypes.sizeof(LossArgs):
    raise ImportError("fastrl_loss_args layout mismatch between libfastrl.so and the binding")
if _lib.fastrl_prune_args_size() != ctypes.sizeof(PruneArgs):
    raise ImportError("fastrl_prune_args layout mismatch between libfastrl.so and the binding")


class FastRLError(RuntimeError):
    pass


def _check(rc, what):
    if rc != 0:
        raise FastRLError(f"{what} failed ({rc}): {_lib.fastrl_last_error().decode()}")


def _p(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _arg(t, dtype, name):
    """Pointer of a caller tensor after checking that the library can read it as the dense
    device array fastrl.h describes (None passes through as NULL)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise FastRLError(f"{name}: expected a device tensor")
    if not t.is_contiguous():
        raise FastRLError(f"{name}: expected a contiguous tensor")
    if dtype is not None and t.dtype != dtype:
        raise FastRLError(f"{name}: expected {dtype}, got {t.dtype}")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _workspace(nbytes, device):
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _dev(t):
    if not t.is_cuda:
        raise FastRLError("expected a device tensor")
    return t


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise FastRLError(f"unsupported dtype {t.dtype}")


def status_names(word):
    return [n for b, n in STATUS_BITS.items() if word & b]


def advantage(rewards, group_off, std_ddof=1, eps=1e-6, drop_uniform=False, status=None):
    """Returns (adv float32[N], class_id int32[N], group_valid uint8[Q])."""
    _dev(rewards)
    Q = group_off.numel() - 1
    N = rewards.numel()
    adv = torch.empty(N, dtype=torch.float32, device=rewards.device)
    cls = torch.empty(N, dtype=torch.int32, device=rewards.device)
    valid = torch.empty(Q, dtype=torch.uint8, device=rewards.device)
    _check(_lib.fastrl_advantage(_arg(rewards, torch.float32, "rewards"),
                                 _arg(group_off, torch.int32, "group_off"), Q, N, std_ddof, eps,
                                 int(bool(drop_uniform)), _p(adv), _p(cls), _p(valid),
                                 _arg(status, torch.int32, "status"), _stream()),
           "fastrl_advantage")
    return adv, cls, valid


def prune(token_ids, traj_tok_off, rewards, group_off, class_id, group_valid, *, V,
          max_group, max_len, ngram_n=1, tau=(4, 5), keep_ratio=0.0, adv=None, group_eps=0.0,
          class_out=False, dp_align=0, status=None):
    """MDAP + budget + compaction.  Returns a dict of device tensors (see fastrl.h).

    ``adv`` (the advantages) sets Alg. 1's traversal order (|A| descending); with
    ``group_eps`` > 0 the classes are the continuous-reward groups |A_i - A_j| < group_eps
    and ``class_id`` is ignored; ``class_out`` adds the class ids used to the result.  The
    plain call (no adv, no group_eps, no class_out) goes through ``fastrl_prune``.
    ``dp_align`` > 1 fills the kept set up to a multiple of that many data-parallel ranks
    (Alg. 1; needs ``adv``)."""
    dev = rewards.device
    Q = group_off.numel() - 1
    N = rewards.numel()
    T_total = token_ids.numel()
    for t, dt, nm in ((token_ids, torch.int32, "token_ids"), (traj_tok_off, torch.int64,
                      "traj_tok_off"), (rewards, torch.float32, "rewards"),
                      (group_off, torch.int32, "group_off"), (class_id, torch.int32, "class_id"),
                      (group_valid, torch.uint8, "group_valid"), (adv, torch.float32, "adv"),
                      (status, torch.int32, "status")):
        _arg(t, dt, nm)
    out = dict(
        keep_mask=torch.empty(N, dtype=torch.uint8, device=dev),
        mdap_count=torch.empty(max(Q, 0), dtype=torch.int32, device=dev),
        kept_traj=torch.empty(max(N, 1), dtype=torch.int32, device=dev),
        kept_tok_off=torch.empty(N + 1, dtype=torch.int64, device=dev),
        tok_src=torch.empty(max(T_total, 1), dtype=torch.int32, device=dev),
        counts=torch.empty(2, dtype=torch.int64, device=dev),
    )
    ws_n = _lib.fastrl_prune_workspace_size(Q, N, T_total, max_group, ngram_n)
    ws = _workspace(ws_n, dev)
    if adv is None and not group_eps and not class_out and dp_align <= 1:
        _check(_lib.fastrl_prune(
            _p(token_ids), _p(traj_tok_off), T_total, _p(rewards), _p(group_off), _p(class_id),
            _p(group_valid), Q, N, max_group, max_len, V, ngram_n, int(tau[0]), int(tau[1]),
            float(keep_ratio), _p(out["keep_mask"]), _p(out["mdap_count"]),
            _p(out["kept_traj"]), _p(out["kept_tok_off"]), _p(out["tok_src"]),
            _p(out["counts"]), _p(status), _p(ws), ws.numel(), _stream()), "fastrl_prune")
        return out
    if class_out:
        out["class_id"] = torch.empty(max(N, 1), dtype=torch.int32, device=dev)
    a = PruneArgs()
    a.token_ids, a.traj_tok_off, a.T_total = _p(token_ids), _p(traj_tok_off), T_total
    a.rewards, a.group_off, a.class_id = _p(rewards), _p(group_off), _p(class_id)
    a.group_valid, a.Q, a.N, a.max_group, a.max_len = _p(group_valid), Q, N, max_group, max_len
    a.V, a.ngram_n, a.tau_num, a.tau_den = V, ngram_n, int(tau[0]), int(tau[1])
    a.keep_ratio = float(keep_ratio)
    a.keep_mask, a.mdap_count = _p(out["keep_mask"]), _p(out["mdap_count"])
    a.kept_traj, a.kept_tok_off = _p(out["kept_traj"]), _p(out["kept_tok_off"])
    a.tok_src, a.counts, a.status = _p(out["tok_src"]), _p(out["counts"]), _p(status)
    a.ws, a.ws_bytes = _p(ws), ws.numel()
    a.adv, a.group_eps = _p(adv), float(group_eps)
    a.class_out = _p(out["class_id"]) if class_out else None
    a.dp_align = int(dp_align)
    _check(_lib.fastrl_prune_ex(ctypes.byref(a), _stream()), "fastrl_prune_ex")
    return out


def token_logprob(hidden, W, token_ids, row_index=None, T=None, status=None):
    """LM-head log-prob of sampled tokens.  Returns (logp float32[T], lse float32[T])."""
    _dev(hidden)
    dt = _dtype_code(hidden)
    d = hidden.shape[1]
    V = W.shape[0]
    for t, dty, nm in ((hidden, hidden.dtype, "hidden"), (W, hidden.dtype, "W"),
                       (token_ids, torch.int32, "token_ids"), (row_index, torch.int32,
                       "row_index"), (status, torch.int32, "status")):
        _arg(t, dty, nm)
    if W.shape[1] != d:
        raise FastRLError("W must be [V, d] with the hidden size of `hidden`")
    if T is None:
        T = row_index.numel() if row_index is not None else hidden.shape[0]
    logp = torch.empty(max(T, 1), dtype=torch.float32, device=hidden.device)
    lse = torch.empty(max(T, 1), dtype=torch.float32, device=hidden.device)
    ws = _workspace(_lib.fastrl_token_logprob_workspace_size(T, d, V, dt), hidden.device)
    _check(_lib.fastrl_token_logprob(_p(hidden), _p(row_index), _p(W), dt, T, d, V,
                                     _p(token_ids), _p(logp), _p(lse), _p(status), _p(ws),
                                     ws.numel(), _stream()), "fastrl_token_logprob")
    return logp[:T], lse[:T]


def token_logprob_noalloc(hidden, W, token_ids, logp, lse=None, row_index=None, T=None,
                          status=None):
    """fastrl_token_logprob_noalloc: the same log-probs with the library's fixed scratch
    and no workspace; the caller passes the outputs (logp, and lse or None), so nothing is
    allocated on this path."""
    _dev(hidden)
    dt = _dtype_code(hidden)
    d = hidden.shape[1]
    V = W.shape[0]
    for t, dty, nm in ((hidden, hidden.dtype, "hidden"), (W, hidden.dtype, "W"),
                       (token_ids, torch.int32, "token_ids"), (row_index, torch.int32,
                       "row_index"), (status, torch.int32, "status"),
                       (logp, torch.float32, "logp"), (lse, torch.float32, "lse")):
        _arg(t, dty, nm)
    if W.shape[1] != d:
        raise FastRLError("W must be [V, d] with the hidden size of `hidden`")
    if T is None:
        T = row_index.numel() if row_index is not None else hidden.shape[0]
    if logp.numel() < T or (lse is not None and lse.numel() < T):
        raise FastRLError("logp / lse must hold T entries")
    _check(_lib.fastrl_token_logprob_noalloc(_p(hidden), _p(row_index), _p(W), dt, T, d, V,
                                             _p(token_ids), _p(logp), _p(lse), _p(status),
                                             _stream()), "fastrl_token_logprob_noalloc")


class LossCall:
    """Prepared arguments of fastrl_policy_loss_fwd_bwd (outputs and workspace are
    allocated once; ``run()`` enqueues the call on the current stream)."""

    def __init__(self, hidden, W, token_ids, old_logp, seq_off, seq_off_host, adv, *,
                 ref_logp=None, seq_index=None, row_index=None, algo="grpo",
                 norm="seq_mean_token_mean", eps_low=0.2, eps_high=0.2, beta=0.0,
                 need_dhidden=True, need_dW=True, dhidden_dtype=None, dW=None,
                 dW_accumulate=False, slab_tokens=0, status=None, T=None,
                 need_entropy=False):
        dev = hidden.device
        dt = _dtype_code(hidden)
        d = hidden.shape[1]
        V = W.shape[0]
        for t, dty, nm in ((hidden, hidden.dtype, "hidden"), (W, hidden.dtype, "W"),
                           (token_ids, torch.int32, "token_ids"),
                           (old_logp, torch.float32, "old_logp"),
                           (ref_logp, torch.float32, "ref_logp"), (seq_off, torch.int64, "seq_off"),
                           (adv, torch.float32, "adv"), (seq_index, torch.int32, "seq_index"),
                           (row_index, torch.int32, "row_index"), (dW, torch.float32, "dW"),
                           (status, torch.int32, "status")):
            _arg(t, dty, nm)
        if W.shape[1] != d:
            raise FastRLError("W must be [V, d] with the hidden size of `hidden`")
        self.seq_off_host = seq_off_host.to(torch.int64).contiguous().cpu()
        S = self.seq_off_host.numel() - 1
        T = int(self.seq_off_host[-1]) if T is None else T
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.stats = torch.zeros(2, dtype=torch.float32, device=dev)
        self.logp = torch.empty(max(T, 1), dtype=torch.float32, device=dev)
        self.lse = torch.empty(max(T, 1), dtype=torch.float32, device=dev)
        self.entropy = (torch.empty(max(T, 1), dtype=torch.float32, device=dev)
                        if need_entropy else None)
        self.entropy_sum = (torch.zeros(1, dtype=torch.float32, device=dev)
                            if need_entropy else None)
        dhd = torch.float32 if dhidden_dtype is None else dhidden_dtype
        self.dhidden = (torch.empty((max(T, 1), d), dtype=dhd, device=dev)
                        if need_dhidden else None)
        if need_dW:
            self.dW = dW if dW is not None else torch.empty((V, d), dtype=torch.float32,
                                                            device=dev)
        else:
            self.dW = None
        self._keep = [hidden, W, token_ids, old_logp, ref_logp, seq_off, adv, seq_index,
                      row_index, status]
        a = LossArgs()
        a.hidden, a.row_index, a.W = _p(hidden), _p(row_index), _p(W)
        a.dtype, a.d, a.V, a.S, a.T = dt, d, V, S, T
        a.token_ids, a.old_logp, a.ref_logp = _p(token_ids), _p(old_logp), _p(ref_logp)
        a.seq_off, a.seq_off_host = _p(seq_off), ctypes.c_void_p(self.seq_off_host.data_ptr())
        a.adv, a.seq_index = _p(adv), _p(seq_index)
        a.algo, a.norm = ALGOS[algo], NORMS[norm]
        a.eps_low, a.eps_high, a.beta = eps_low, eps_high, beta
        a.loss, a.logp, a.lse = _p(self.loss), _p(self.logp), _p(self.lse)
        a.dhidden = _p(self.dhidden)
        a.dhidden_dtype = _dtype_code(self.dhidden) if self.dhidden is not None else F32
        a.dW = _p(self.dW)
        a.dW_accumulate = int(bool(dW_accumulate))
        a.stats = _p(self.stats)
        a.entropy, a.entropy_sum = _p(self.entropy), _p(self.entropy_sum)
        a.slab_tokens = int(slab_tokens)
        a.status = _p(status)
        n = _lib.fastrl_policy_loss_workspace_size(ctypes.byref(a))
        if n == 0:
            _check(-2, "fastrl_policy_loss_workspace_size")
        self.ws = _workspace(n, dev)
        a.ws, a.ws_bytes = _p(self.ws), self.ws.numel()
        self.args = a
        self.T = T

    def run(self):
        _check(_lib.fastrl_policy_loss_fwd_bwd(ctypes.byref(self.args), _stream()),
               "fastrl_policy_loss_fwd_bwd")
        return self

    def slab_plan(self):
        """(first sequence of each slab followed by S, largest slab's token count)."""
        return slab_plan(self.args)


def slab_plan(args):
    """The slabs fastrl_policy_loss_fwd_bwd runs for a LossArgs (host only): returns
    (list of each slab's first sequence followed by S, largest slab's token count)."""
    tc = _i64()
    n = _lib.fastrl_policy_loss_slab_plan(ctypes.byref(args), None, 0, ctypes.byref(tc))
    _check(min(n, 0), "fastrl_policy_loss_slab_plan")
    buf = (ctypes.c_int32 * (n + 1))()
    _lib.fastrl_policy_loss_slab_plan(ctypes.byref(args), buf, n + 1, None)
    return list(buf), tc.value


def policy_loss_fwd_bwd(*args, **kw):
    """One call of fastrl_policy_loss_fwd_bwd; returns the LossCall holding the outputs
    (loss, logp, lse, dhidden, dW, stats, and entropy / entropy_sum with need_entropy)."""
    return LossCall(*args, **kw).run()


def adamw_step(theta, grad, m, v, *, step, lr=1e-6, betas=(0.9, 0.999), eps=1e-8,
               weight_decay=1e-2, grad_scale=1.0, w_bf16=None, status=None):
    """In-place AdamW update of float32 ``theta``, ``m``, ``v`` from ``grad`` (e.g. dW);
    optionally writes the bfloat16 copy ``w_bf16``.  ``step`` is 1-based."""
    n = theta.numel()
    for t, nm in ((theta, "theta"), (grad, "grad"), (m, "m"), (v, "v")):
        _arg(t, torch.float32, nm)
        if t.numel() != n:
            raise FastRLError(f"{nm}: expected {n} elements")
    _arg(w_bf16, torch.bfloat16, "w_bf16")
    _arg(status, torch.int32, "status")
    if w_bf16 is not None and w_bf16.numel() != n:
        raise FastRLError(f"w_bf16: expected {n} elements")
    _check(_lib.fastrl_adamw_step(_p(theta), _p(w_bf16), _p(grad), _p(m), _p(v), n, int(step),
                                  float(lr), float(betas[0]), float(betas[1]), float(eps),
                                  float(weight_decay), float(grad_scale), _p(status),
                                  _stream()), "fastrl_adamw_step")


class ARS:
    """Adaptive Rollout Sampling controller (host only); ``state`` is a plain struct."""

    def __init__(self, G1, total_steps, steps_per_epoch):
        self.state = ARSState()
        _check(_lib.fastrl_ars_init(ctypes.byref(self.state), G1, total_steps,
                                    steps_per_epoch), "fastrl_ars_init")

    def next_n(self):
        return int(_lib.fastrl_ars_next_n(ctypes.byref(self.state)))

    def observe(self, counts, valid=None):
        c = (ctypes.c_int32 * len(counts))(*[int(x) for x in counts])
        v = None if valid is None else (ctypes.c_uint8 * len(valid))(*[int(x) for x in valid])
        _check(_lib.fastrl_ars_observe(ctypes.byref(self.state), c, v, len(counts)),
               "fastrl_ars_observe")

    def to_bytes(self):
        return bytes(self.state)

    @classmethod
    def from_bytes(cls, b):
        obj = cls.__new__(cls)
        obj.state = ARSState.from_buffer_copy(b)
        return obj


def profile_enable(on=True):
    _lib.fastrl_profile_enable(int(bool(on)))


def profile_reset():
    _lib.fastrl_profile_reset()


def profile_read(kind):
    ms, n, fl = _f64(), _i64(), _f64()
    _check(_lib.fastrl_profile_read(kind, ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl)),
           "fastrl_profile_read")
    return ms.value, n.value, fl.value


def hot_path_step(rewards, group_off, token_ids, traj_tok_off, hidden, W, old_logp,
                  ref_logp=None, *, V, max_group, max_len, algo="grpo",
                  norm="seq_mean_token_mean", eps_low=0.2, eps_high=0.2, beta=0.0,
                  ngram_n=1, tau=(4, 5), keep_ratio=0.0, drop_uniform=False,
                  need_dhidden=True, need_dW=True, slab_tokens=0, status=None,
                  dhidden_dtype=None, group_eps=0.0, dp_align=0):
    """advantage -> prune + compaction -> (one device->host read of the kept counts and
    offsets) -> loss forward/backward on the kept tokens.  Returns a dict.  ``group_eps``
    > 0 prunes under continuous-reward groups |A_i - A_j| < group_eps."""
    adv, cls, valid = advantage(rewards, group_off, drop_uniform=drop_uniform, status=status)
    pr = prune(token_ids, traj_tok_off, rewards, group_off, cls, valid, V=V,
               max_group=max_group, max_len=max_len, ngram_n=ngram_n, tau=tau,
               keep_ratio=keep_ratio, status=status,
               adv=adv if (group_eps or dp_align > 1) else None, group_eps=group_eps,
               dp_align=dp_align)
    counts = pr["counts"].cpu()
    n_kept, t_kept = int(counts[0]), int(counts[1])
    koff_host = pr["kept_tok_off"][:n_kept + 1].cpu()
    call = LossCall(hidden, W, token_ids, old_logp, pr["kept_tok_off"], koff_host, adv,
                    ref_logp=ref_logp, seq_index=pr["kept_traj"], row_index=pr["tok_src"],
                    algo=algo, norm=norm, eps_low=eps_low, eps_high=eps_high, beta=beta,
                    need_dhidden=need_dhidden, need_dW=need_dW, slab_tokens=slab_tokens,
                    status=status, T=t_kept, dhidden_dtype=dhidden_dtype).run()
    return dict(adv=adv, class_id=cls, group_valid=valid, prune=pr, n_kept=n_kept,
                t_kept=t_kept, kept_tok_off_host=koff_host, call=call)
