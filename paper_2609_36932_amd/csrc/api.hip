// C ABI of libfastrl: argument validation, error text, workspace queries, kernel timing,
// and the host-only Adaptive Rollout Sampling controller (Sec. 3.3; Alg. 1 Phase 1).
#include <atomic>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

namespace fastrl {

int launch_advantage(const float*, const int32_t*, int32_t, int32_t, int32_t, float, int32_t,
                     float*, int32_t*, uint8_t*, int32_t*, hipStream_t);
size_t prune_workspace(int32_t Q, int32_t N, int64_t T_total, int32_t max_group);
int launch_prune(const int32_t*, const int64_t*, int64_t, const float*, const int32_t*,
                 const int32_t*, const float*, double, const uint8_t*, int32_t, int32_t,
                 int32_t, int32_t, int32_t, int32_t, int32_t, int32_t, double, uint8_t*,
                 int32_t*, int32_t*, int32_t, int32_t*, int64_t*, int32_t*, int64_t*, int32_t*,
                 void*, hipStream_t);
size_t token_logprob_workspace(int64_t T, int32_t d, int32_t V, int32_t dtype);
int run_token_logprob_noalloc(const void*, const int32_t*, const void*, int32_t, int64_t,
                              int32_t, int32_t, const int32_t*, float*, float*, int32_t*,
                              hipStream_t);
size_t token_logprob_noalloc_scratch_bytes();
int64_t token_logprob_noalloc_chunk(int32_t V);
int run_token_logprob(const void*, const int32_t*, const void*, int32_t, int64_t, int32_t,
                      int32_t, const int32_t*, float*, float*, int32_t*, void*, hipStream_t);
size_t policy_loss_workspace(const fastrl_loss_args& a);
int policy_loss_slab_plan(const fastrl_loss_args& a, int32_t* seq_begin, int32_t capacity,
                          int64_t* tc_max);
int launch_adamw(float* theta, uint16_t* wbf, const float* grad, float* mom, float* var,
                 int64_t n, int64_t step, float lr, float beta1, float beta2, float eps,
                 float weight_decay, float grad_scale, int32_t* status, hipStream_t stream);
int run_policy_loss(const fastrl_loss_args& a, hipStream_t stream);

static thread_local std::string g_err;
void set_error(const std::string& msg) { g_err = msg; }
void clear_error() { g_err.clear(); }

// ---- kernel timing recorder ------------------------------------------------------------
struct ProfRec {
  int kind;
  double flops;
  hipEvent_t a, b;
};
static std::atomic<bool> g_prof_on{false};
static std::mutex g_prof_mu;  // guards g_prof and g_ev_pool
static std::vector<ProfRec> g_prof;
static std::vector<hipEvent_t> g_ev_pool;

static hipEvent_t take_event() {
  if (!g_ev_pool.empty()) {
    hipEvent_t e = g_ev_pool.back();
    g_ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

ProfScope::ProfScope(int k, hipStream_t s, double f) : kind(k), stream(s), flops(f) {
  if (!g_prof_on.load(std::memory_order_relaxed) || k < 0) return;
  std::lock_guard<std::mutex> lock(g_prof_mu);
  hipEvent_t e = take_event();
  if (e && hipEventRecord(e, s) == hipSuccess) ev0 = e;
}
ProfScope::~ProfScope() {
  if (!ev0) return;
  std::lock_guard<std::mutex> lock(g_prof_mu);
  hipEvent_t e = take_event();
  if (e && hipEventRecord(e, stream) == hipSuccess)
    g_prof.push_back(ProfRec{kind, flops, static_cast<hipEvent_t>(ev0), e});
}

static bool aligned256(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 255u) == 0; }
static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace fastrl

using namespace fastrl;

extern "C" {

const char* fastrl_last_error(void) { return g_err.c_str(); }
int fastrl_version(void) { return 10100; }

int fastrl_advantage(const float* rewards, const int32_t* group_off, int32_t Q, int32_t N,
                     int32_t std_ddof, float eps, int32_t drop_uniform, float* adv,
                     int32_t* class_id, uint8_t* group_valid, int32_t* status,
                     hipStream_t stream) {
  clear_error();
  FR_CHECK_ARG(Q >= 0 && N >= 0, FASTRL_ERR_SHAPE, "fastrl_advantage: Q and N must be >= 0");
  FR_CHECK_ARG(std_ddof == 0 || std_ddof == 1, FASTRL_ERR_VALUE,
               "fastrl_advantage: std_ddof must be 0 or 1");
  FR_CHECK_ARG(eps >= 0.0f && std::isfinite(eps), FASTRL_ERR_VALUE,
               "fastrl_advantage: eps must be finite and >= 0");
  if (Q == 0) return FASTRL_OK;
  FR_CHECK_ARG(group_off && group_valid, FASTRL_ERR_NULL_PTR,
               "fastrl_advantage: group_off / group_valid is NULL");
  FR_CHECK_ARG(N == 0 || (rewards && adv && class_id), FASTRL_ERR_NULL_PTR,
               "fastrl_advantage: rewards / adv / class_id is NULL");
  return launch_advantage(rewards, group_off, Q, N, std_ddof, eps, drop_uniform, adv, class_id,
                          group_valid, status, stream);
}

size_t fastrl_prune_workspace_size(int32_t Q, int32_t N, int64_t T_total, int32_t max_group,
                                   int32_t ngram_n) {
  (void)ngram_n;
  if (Q < 0 || N < 0 || T_total < 0 || max_group < 1) return 0;
  return prune_workspace(Q, N, T_total, max_group);
}

static int check_and_prune(const fastrl_prune_args& a, hipStream_t stream) {
  const char* fn = "fastrl_prune";
  FR_CHECK_ARG(a.Q >= 0 && a.N >= 0 && a.T_total >= 0, FASTRL_ERR_SHAPE,
               std::string(fn) + ": Q, N, T_total must be >= 0");
  FR_CHECK_ARG(a.T_total < (int64_t(1) << 31), FASTRL_ERR_SHAPE,
               std::string(fn) + ": T_total must be < 2^31");
  FR_CHECK_ARG(a.max_group >= 1 && a.max_group <= 256, FASTRL_ERR_SHAPE,
               std::string(fn) + ": max_group must be in [1, 256]");
  FR_CHECK_ARG(a.max_len >= 0 && a.max_len <= 16384, FASTRL_ERR_SHAPE,
               std::string(fn) + ": max_len must be in [0, 16384]");
  FR_CHECK_ARG(a.V >= 1 && a.V < (1 << 21), FASTRL_ERR_VALUE,
               std::string(fn) + ": V must be in [1, 2^21)");
  FR_CHECK_ARG(a.ngram_n >= 1 && a.ngram_n <= 3, FASTRL_ERR_VALUE,
               std::string(fn) + ": ngram_n must be 1, 2 or 3");
  FR_CHECK_ARG(a.tau_num >= 0 && a.tau_den > 0, FASTRL_ERR_VALUE,
               std::string(fn) + ": need tau_num >= 0 and tau_den > 0");
  FR_CHECK_ARG(a.keep_ratio >= 0.0 && a.keep_ratio <= 1.0, FASTRL_ERR_VALUE,
               std::string(fn) + ": keep_ratio must be in [0, 1]");
  FR_CHECK_ARG(a.group_eps >= 0.0 && std::isfinite(a.group_eps), FASTRL_ERR_VALUE,
               std::string(fn) + ": group_eps must be finite and >= 0");
  FR_CHECK_ARG(a.traj_tok_off && a.kept_tok_off && a.counts, FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": traj_tok_off / kept_tok_off / counts is NULL");
  FR_CHECK_ARG(a.N == 0 || (a.keep_mask && a.kept_traj && a.rewards), FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": keep_mask / kept_traj / rewards is NULL");
  FR_CHECK_ARG(a.N == 0 || a.group_eps > 0.0 || a.class_id, FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": class_id is NULL (needed unless group_eps > 0)");
  FR_CHECK_ARG(a.N == 0 || !(a.group_eps > 0.0) || a.adv, FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": group_eps > 0 needs adv");
  FR_CHECK_ARG(a.dp_align >= 0 && a.dp_align <= 4096, FASTRL_ERR_VALUE,
               std::string(fn) + ": dp_align must be in [0, 4096]");
  FR_CHECK_ARG(a.N == 0 || a.dp_align <= 1 || a.adv, FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": dp_align > 1 needs adv");
  FR_CHECK_ARG(a.Q == 0 || (a.group_off && a.mdap_count), FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": group_off / mdap_count is NULL");
  FR_CHECK_ARG(a.T_total == 0 || (a.token_ids && a.tok_src), FASTRL_ERR_NULL_PTR,
               std::string(fn) + ": token_ids / tok_src is NULL");
  const size_t need = prune_workspace(a.Q, a.N, a.T_total, a.max_group);
  FR_CHECK_ARG(a.ws && aligned256(a.ws) && a.ws_bytes >= need, FASTRL_ERR_WORKSPACE,
               std::string(fn) + ": workspace missing, misaligned or smaller than " +
                   std::to_string(need) + " bytes");
  return launch_prune(a.token_ids, a.traj_tok_off, a.T_total, a.rewards, a.group_off,
                      a.class_id, a.adv, a.group_eps, a.group_valid, a.Q, a.N, a.max_group,
                      a.max_len, a.V, a.ngram_n, a.tau_num, a.tau_den, a.keep_ratio,
                      a.keep_mask, a.mdap_count, a.class_out, a.dp_align, a.kept_traj,
                      a.kept_tok_off,
                      a.tok_src, a.counts, a.status, a.ws, stream);
}

int fastrl_prune(const int32_t* token_ids, const int64_t* traj_tok_off, int64_t T_total,
                 const float* rewards, const int32_t* group_off, const int32_t* class_id,
                 const uint8_t* group_valid, int32_t Q, int32_t N, int32_t max_group,
                 int32_t max_len, int32_t V, int32_t ngram_n, int32_t tau_num,
                 int32_t tau_den, double keep_ratio, uint8_t* keep_mask,
                 int32_t* mdap_count, int32_t* kept_traj, int64_t* kept_tok_off,
                 int32_t* tok_src, int64_t* counts, int32_t* status, void* ws,
                 size_t ws_bytes, hipStream_t stream) {
  clear_error();
  fastrl_prune_args a{};
  a.token_ids = token_ids; a.traj_tok_off = traj_tok_off; a.T_total = T_total;
  a.rewards = rewards; a.group_off = group_off; a.class_id = class_id;
  a.group_valid = group_valid; a.Q = Q; a.N = N; a.max_group = max_group;
  a.max_len = max_len; a.V = V; a.ngram_n = ngram_n; a.tau_num = tau_num;
  a.tau_den = tau_den; a.keep_ratio = keep_ratio; a.keep_mask = keep_mask;
  a.mdap_count = mdap_count; a.kept_traj = kept_traj; a.kept_tok_off = kept_tok_off;
  a.tok_src = tok_src; a.counts = counts; a.status = status; a.ws = ws; a.ws_bytes = ws_bytes;
  return check_and_prune(a, stream);
}

size_t fastrl_prune_args_size(void) { return sizeof(fastrl_prune_args); }

int fastrl_prune_ex(const fastrl_prune_args* a, hipStream_t stream) {
  clear_error();
  FR_CHECK_ARG(a != nullptr, FASTRL_ERR_NULL_PTR, "fastrl_prune_ex: args is NULL");
  return check_and_prune(*a, stream);
}

size_t fastrl_token_logprob_workspace_size(int64_t T, int32_t d, int32_t V, int32_t dtype) {
  if (T < 0 || d < 1 || V < 1) return 0;
  return token_logprob_workspace(T, d, V, dtype);
}

int fastrl_token_logprob(const void* hidden, const int32_t* row_index, const void* W,
                         int32_t dtype, int64_t T, int32_t d, int32_t V,
                         const int32_t* token_ids, float* logp, float* lse,
                         int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream) {
  clear_error();
  FR_CHECK_ARG(dtype == FASTRL_F32 || dtype == FASTRL_BF16, FASTRL_ERR_DTYPE,
               "fastrl_token_logprob: dtype must be FASTRL_F32 or FASTRL_BF16");
  FR_CHECK_ARG(T >= 0 && d >= 8 && d % 8 == 0 && V >= 1, FASTRL_ERR_SHAPE,
               "fastrl_token_logprob: need T >= 0, d a positive multiple of 8, V >= 1");
  FR_CHECK_ARG(T < (int64_t(1) << 31) && V < (1 << 30), FASTRL_ERR_SHAPE,
               "fastrl_token_logprob: T or V too large");
  if (T == 0) return FASTRL_OK;
  FR_CHECK_ARG(hidden && W && token_ids && logp, FASTRL_ERR_NULL_PTR,
               "fastrl_token_logprob: hidden / W / token_ids / logp is NULL");
  FR_CHECK_ARG(aligned16(hidden) && aligned16(W), FASTRL_ERR_VALUE,
               "fastrl_token_logprob: hidden and W must be 16-byte aligned");
  const size_t need = token_logprob_workspace(T, d, V, dtype);
  FR_CHECK_ARG(ws && aligned256(ws) && ws_bytes >= need, FASTRL_ERR_WORKSPACE,
               "fastrl_token_logprob: workspace missing, misaligned or smaller than " +
                   std::to_string(need) + " bytes");
  return run_token_logprob(hidden, row_index, W, dtype, T, d, V, token_ids, logp, lse, status,
                           ws, stream);
}

int fastrl_token_logprob_noalloc(const void* hidden, const int32_t* row_index, const void* W,
                                 int32_t dtype, int64_t T, int32_t d, int32_t V,
                                 const int32_t* token_ids, float* logp, float* lse,
                                 int32_t* status, hipStream_t stream) {
  clear_error();
  FR_CHECK_ARG(dtype == FASTRL_F32 || dtype == FASTRL_BF16, FASTRL_ERR_DTYPE,
               "fastrl_token_logprob_noalloc: dtype must be FASTRL_F32 or FASTRL_BF16");
  FR_CHECK_ARG(T >= 0 && d >= 8 && d % 8 == 0 && V >= 1, FASTRL_ERR_SHAPE,
               "fastrl_token_logprob_noalloc: need T >= 0, d a positive multiple of 8, V >= 1");
  FR_CHECK_ARG(T < (int64_t(1) << 31) && V < (1 << 30), FASTRL_ERR_SHAPE,
               "fastrl_token_logprob_noalloc: T or V too large");
  if (T > 0) {
    FR_CHECK_ARG(hidden && W && token_ids && logp, FASTRL_ERR_NULL_PTR,
                 "fastrl_token_logprob_noalloc: hidden / W / token_ids / logp is NULL");
    FR_CHECK_ARG(aligned16(hidden) && aligned16(W), FASTRL_ERR_VALUE,
                 "fastrl_token_logprob_noalloc: hidden and W must be 16-byte aligned");
  }
  return run_token_logprob_noalloc(hidden, row_index, W, dtype, T, d, V, token_ids, logp, lse,
                                   status, stream);
}

size_t fastrl_token_logprob_noalloc_scratch_bytes(void) {
  return token_logprob_noalloc_scratch_bytes();
}

int64_t fastrl_token_logprob_noalloc_max_chunk(int32_t V) {
  return V >= 1 ? token_logprob_noalloc_chunk(V) : 0;
}

static int check_loss_args(const fastrl_loss_args* a, bool need_ws) {
  FR_CHECK_ARG(a != nullptr, FASTRL_ERR_NULL_PTR, "fastrl_policy_loss: args is NULL");
  FR_CHECK_ARG(a->dtype == FASTRL_F32 || a->dtype == FASTRL_BF16, FASTRL_ERR_DTYPE,
               "fastrl_policy_loss: dtype must be FASTRL_F32 or FASTRL_BF16");
  FR_CHECK_ARG(a->dhidden == nullptr || a->dhidden_dtype == FASTRL_F32 ||
                   a->dhidden_dtype == FASTRL_BF16,
               FASTRL_ERR_DTYPE, "fastrl_policy_loss: bad dhidden_dtype");
  FR_CHECK_ARG(a->d >= 8 && a->d % 8 == 0 && a->V >= 1 && a->V < (1 << 30) && a->S >= 0 &&
                   a->T >= 0 && a->T < (int64_t(1) << 31),
               FASTRL_ERR_SHAPE,
               "fastrl_policy_loss: need d a positive multiple of 8, V >= 1, S >= 0, 0 <= T < 2^31");
  FR_CHECK_ARG(a->algo >= FASTRL_GRPO && a->algo <= FASTRL_GSPO, FASTRL_ERR_VALUE,
               "fastrl_policy_loss: unknown algo");
  FR_CHECK_ARG(a->norm == FASTRL_NORM_SEQ_MEAN_TOKEN_MEAN || a->norm == FASTRL_NORM_TOKEN_MEAN,
               FASTRL_ERR_VALUE, "fastrl_policy_loss: unknown norm");
  FR_CHECK_ARG(std::isfinite(a->eps_low) && std::isfinite(a->eps_high) && a->eps_low >= 0 &&
                   a->eps_high >= 0 && a->eps_low < 1,
               FASTRL_ERR_VALUE, "fastrl_policy_loss: need 0 <= eps_low < 1, eps_high >= 0");
  FR_CHECK_ARG(std::isfinite(a->beta), FASTRL_ERR_VALUE, "fastrl_policy_loss: beta not finite");
  FR_CHECK_ARG(a->slab_tokens >= 0, FASTRL_ERR_VALUE, "fastrl_policy_loss: slab_tokens < 0");
  FR_CHECK_ARG(a->seq_off_host && a->seq_off && a->loss, FASTRL_ERR_NULL_PTR,
               "fastrl_policy_loss: seq_off / seq_off_host / loss is NULL");
  FR_CHECK_ARG(a->seq_off_host[0] == 0 && a->seq_off_host[a->S] == a->T, FASTRL_ERR_SHAPE,
               "fastrl_policy_loss: seq_off_host must start at 0 and end at T");
  for (int32_t i = 0; i < a->S; ++i)
    FR_CHECK_ARG(a->seq_off_host[i + 1] >= a->seq_off_host[i], FASTRL_ERR_SHAPE,
                 "fastrl_policy_loss: seq_off_host is not monotone");
  if (a->T > 0) {
    FR_CHECK_ARG(a->hidden && a->W && a->token_ids && a->old_logp, FASTRL_ERR_NULL_PTR,
                 "fastrl_policy_loss: hidden / W / token_ids / old_logp is NULL");
    FR_CHECK_ARG(aligned16(a->hidden) && aligned16(a->W), FASTRL_ERR_VALUE,
                 "fastrl_policy_loss: hidden and W must be 16-byte aligned");
    FR_CHECK_ARG(aligned16(a->dW), FASTRL_ERR_VALUE,
                 "fastrl_policy_loss: dW must be 16-byte aligned");
  }
  FR_CHECK_ARG(a->S == 0 || a->adv, FASTRL_ERR_NULL_PTR, "fastrl_policy_loss: adv is NULL");
  FR_CHECK_ARG(a->beta == 0.0f || a->ref_logp || a->T == 0, FASTRL_ERR_NULL_PTR,
               "fastrl_policy_loss: ref_logp is NULL while beta != 0");
  if (need_ws) {
    const size_t need = policy_loss_workspace(*a);
    FR_CHECK_ARG(a->ws && aligned256(a->ws) && a->ws_bytes >= need, FASTRL_ERR_WORKSPACE,
                 "fastrl_policy_loss: workspace missing, misaligned or smaller than " +
                     std::to_string(need) + " bytes");
  }
  return FASTRL_OK;
}

size_t fastrl_loss_args_size(void) { return sizeof(fastrl_loss_args); }

size_t fastrl_policy_loss_workspace_size(const fastrl_loss_args* args) {
  clear_error();
  if (check_loss_args(args, false) != FASTRL_OK) return 0;
  return policy_loss_workspace(*args);
}

int fastrl_policy_loss_slab_plan(const fastrl_loss_args* args, int32_t* seq_begin_host,
                                 int32_t capacity, int64_t* max_slab_tokens) {
  clear_error();
  const int rc = check_loss_args(args, false);
  if (rc != FASTRL_OK) return rc;
  return policy_loss_slab_plan(*args, seq_begin_host, capacity, max_slab_tokens);
}

int fastrl_policy_loss_fwd_bwd(const fastrl_loss_args* args, hipStream_t stream) {
  clear_error();
  const int rc = check_loss_args(args, true);
  if (rc != FASTRL_OK) return rc;
  return run_policy_loss(*args, stream);
}

// ---- ARS -------------------------------------------------------------------------------
int fastrl_ars_init(fastrl_ars_state* st, int32_t G1, int64_t total_steps,
                    int64_t steps_per_epoch) {
  clear_error();
  FR_CHECK_ARG(st != nullptr, FASTRL_ERR_NULL_PTR, "fastrl_ars_init: state is NULL");
  FR_CHECK_ARG(G1 >= 2 && total_steps >= 1 && steps_per_epoch >= 1, FASTRL_ERR_VALUE,
               "fastrl_ars_init: need G1 >= 2, total_steps >= 1, steps_per_epoch >= 1");
  std::memset(st, 0, sizeof(*st));
  st->G = G1;
  st->total_steps = total_steps;
  st->steps_per_epoch = steps_per_epoch;
  st->G_ref = NAN;
  st->G_t = NAN;
  return FASTRL_OK;
}

int32_t fastrl_ars_next_n(const fastrl_ars_state* st) {
  if (!st) return 0;
  if (!std::isnan(st->G_t) && !std::isnan(st->G_ref) && st->G_t < st->G_ref) {
    const double x = std::fmin(double(st->G) - (st->G_ref - st->G_t), double(st->G));
    const double r = std::nearbyint(x);  // default rounding mode: half to even
    return int32_t(std::fmax(r, 2.0));
  }
  return st->G;
}

int fastrl_ars_observe(fastrl_ars_state* st, const int32_t* counts_host,
                       const uint8_t* valid_host, int32_t Q) {
  clear_error();
  FR_CHECK_ARG(st != nullptr, FASTRL_ERR_NULL_PTR, "fastrl_ars_observe: state is NULL");
  FR_CHECK_ARG(Q >= 0, FASTRL_ERR_SHAPE, "fastrl_ars_observe: Q < 0");
  FR_CHECK_ARG(Q == 0 || counts_host, FASTRL_ERR_NULL_PTR, "fastrl_ars_observe: counts is NULL");
  int64_t sum = 0, n = 0;
  int32_t mx = 0;
  for (int32_t q = 0; q < Q; ++q) {
    if (valid_host && !valid_host[q]) continue;
    sum += counts_host[q];
    mx = (n == 0 || counts_host[q] > mx) ? counts_host[q] : mx;
    ++n;
  }
  st->step += 1;
  if (n > 0) {
    st->sum_mean += double(sum) / double(n);
    st->sum_max += double(mx);
    st->n_buf += 1;
  }
  if (st->step % st->steps_per_epoch == 0) {
    if (st->n_buf > 0) {
      const double bm = st->sum_mean / double(st->n_buf);
      const double bM = st->sum_max / double(st->n_buf);
      const double alpha = double(st->step) / double(st->total_steps);
      st->G_t = alpha * bm + (1.0 - alpha) * bM;
      if (std::isnan(st->G_ref)) st->G_ref = (bm + bM) / 2.0;
    }
    st->sum_mean = 0.0;
    st->sum_max = 0.0;
    st->n_buf = 0;
  }
  return FASTRL_OK;
}

// ---- kernel timing ---------------------------------------------------------------------
int fastrl_profile_enable(int32_t on) {
  g_prof_on.store(on != 0, std::memory_order_relaxed);
  return FASTRL_OK;
}

int fastrl_profile_reset(void) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  for (auto& r : g_prof) {
    g_ev_pool.push_back(r.a);
    g_ev_pool.push_back(r.b);
  }
  g_prof.clear();
  return FASTRL_OK;
}

int fastrl_profile_read(int32_t kind, double* total_ms, int64_t* launches, double* flops) {
  clear_error();
  FR_CHECK_ARG(total_ms && launches && flops, FASTRL_ERR_NULL_PTR,
               "fastrl_profile_read: NULL output");
  double ms = 0.0, fl = 0.0;
  int64_t n = 0;
  std::lock_guard<std::mutex> lock(g_prof_mu);
  for (auto& r : g_prof) {
    if (r.kind != kind) continue;
    FR_HIP(hipEventSynchronize(r.b));
    float t = 0.0f;
    FR_HIP(hipEventElapsedTime(&t, r.a, r.b));
    ms += t;
    fl += r.flops;
    ++n;
  }
  *total_ms = ms;
  *launches = n;
  *flops = fl;
  return FASTRL_OK;
}

int fastrl_adamw_step(float* theta, uint16_t* w_bf16, const float* grad, float* m, float* v,
                      int64_t n, int64_t step, float lr, float beta1, float beta2, float eps,
                      float weight_decay, float grad_scale, int32_t* status,
                      hipStream_t stream) {
  clear_error();
  FR_CHECK_ARG(n >= 0 && step >= 1, FASTRL_ERR_SHAPE, "fastrl_adamw_step: need n >= 0, step >= 1");
  FR_CHECK_ARG(std::isfinite(lr) && lr >= 0 && std::isfinite(eps) && eps >= 0 &&
                   std::isfinite(weight_decay) && weight_decay >= 0 &&
                   std::isfinite(grad_scale) && beta1 >= 0 && beta1 < 1 && beta2 >= 0 &&
                   beta2 < 1,
               FASTRL_ERR_VALUE,
               "fastrl_adamw_step: need finite lr, eps, weight_decay, grad_scale >= 0 (except "
               "grad_scale) and betas in [0, 1)");
  if (n == 0) return FASTRL_OK;
  FR_CHECK_ARG(theta && grad && m && v, FASTRL_ERR_NULL_PTR,
               "fastrl_adamw_step: theta / grad / m / v is NULL");
  auto al = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; };
  FR_CHECK_ARG(al(theta, 16) && al(grad, 16) && al(m, 16) && al(v, 16) &&
                   (w_bf16 == nullptr || al(w_bf16, 8)),
               FASTRL_ERR_VALUE,
               "fastrl_adamw_step: theta / grad / m / v must be 16-byte aligned, w_bf16 8-byte");
  return launch_adamw(theta, w_bf16, grad, m, v, n, step, lr, beta1, beta2, eps, weight_decay,
                      grad_scale, status, stream);
}

}  // extern "C"
