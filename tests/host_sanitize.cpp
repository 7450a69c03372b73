// Host-side driver for the AddressSanitizer / UndefinedBehaviorSanitizer build of libfastrl's
// C ABI (built by tests/test_host_sanitizers.py with the sanitizers on the host code only).
// It needs no GPU: it runs every host-side validation path that returns before anything is
// enqueued, the workspace-size queries, the slab planner of the loss call on many random
// length mixes, and the adaptive rollout sampling controller, and checks their results.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "../include/fastrl.h"

static int g_fail = 0;
#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      std::fprintf(stderr, "CHECK failed line %d: %s (%s)\n", __LINE__, #cond, \
                   fastrl_last_error());                              \
      ++g_fail;                                                       \
    }                                                                 \
  } while (0)

static void* dummy() { return reinterpret_cast<void*>(uintptr_t(256)); }

static void validation_paths() {
  // advantage: negative sizes, bad ddof, NULL arrays; the empty call succeeds
  CHECK(fastrl_advantage(nullptr, nullptr, -1, 0, 1, 1e-6f, 0, nullptr, nullptr, nullptr,
                         nullptr, nullptr) == FASTRL_ERR_SHAPE);
  CHECK(fastrl_advantage(nullptr, nullptr, 1, 1, 2, 1e-6f, 0, nullptr, nullptr, nullptr,
                         nullptr, nullptr) == FASTRL_ERR_VALUE);
  CHECK(fastrl_advantage(nullptr, nullptr, 1, 1, 1, 1e-6f, 0, nullptr, nullptr, nullptr,
                         nullptr, nullptr) == FASTRL_ERR_NULL_PTR);
  CHECK(fastrl_advantage(nullptr, nullptr, 0, 0, 1, 1e-6f, 0, nullptr, nullptr, nullptr,
                         nullptr, nullptr) == FASTRL_OK);
  // prune: out-of-range n, V, tau, group size, keep ratio; NULL arrays
  auto prune = [](int32_t n, int32_t V, int32_t tden, int32_t G, double keep) {
    return fastrl_prune(nullptr, nullptr, 10, nullptr, nullptr, nullptr, nullptr, 2, 16, G, 64,
                        V, n, 4, tden, keep, nullptr, nullptr, nullptr, nullptr, nullptr,
                        nullptr, nullptr, nullptr, 0, nullptr);
  };
  CHECK(prune(4, 1000, 5, 8, 0.5) == FASTRL_ERR_VALUE);
  CHECK(prune(1, 1 << 21, 5, 8, 0.5) == FASTRL_ERR_VALUE);
  CHECK(prune(1, 1000, 0, 8, 0.5) == FASTRL_ERR_VALUE);
  CHECK(prune(1, 1000, 5, 300, 0.5) == FASTRL_ERR_SHAPE);
  CHECK(prune(1, 1000, 5, 8, 1.5) == FASTRL_ERR_VALUE);
  CHECK(prune(1, 1000, 5, 8, 0.5) == FASTRL_ERR_NULL_PTR);
  CHECK(fastrl_prune_ex(nullptr, nullptr) == FASTRL_ERR_NULL_PTR);
  fastrl_prune_args pa;
  std::memset(&pa, 0, sizeof(pa));
  pa.T_total = 10; pa.Q = 2; pa.N = 16; pa.max_group = 8; pa.max_len = 64; pa.V = 1000;
  pa.ngram_n = 1; pa.tau_num = 4; pa.tau_den = 5; pa.keep_ratio = 0.5; pa.group_eps = NAN;
  CHECK(fastrl_prune_ex(&pa, nullptr) == FASTRL_ERR_VALUE);
  CHECK(fastrl_prune_args_size() == sizeof(fastrl_prune_args));
  CHECK(fastrl_prune_workspace_size(64, 512, 300000, 8, 1) > 0);
  // token log-prob: bad dtype, bad d, NULL arrays, misaligned pointers, small workspace
  int32_t dt = 7;
  CHECK(fastrl_token_logprob(dummy(), nullptr, dummy(), dt, 4, 64, 100, (int32_t*)dummy(),
                             (float*)dummy(), nullptr, nullptr, dummy(), 1 << 20,
                             nullptr) == FASTRL_ERR_DTYPE);
  CHECK(fastrl_token_logprob(dummy(), nullptr, dummy(), FASTRL_BF16, 4, 12, 100,
                             (int32_t*)dummy(), (float*)dummy(), nullptr, nullptr, dummy(),
                             1 << 20, nullptr) == FASTRL_ERR_SHAPE);
  CHECK(fastrl_token_logprob(nullptr, nullptr, dummy(), FASTRL_BF16, 4, 64, 100,
                             (int32_t*)dummy(), (float*)dummy(), nullptr, nullptr, dummy(),
                             1 << 20, nullptr) == FASTRL_ERR_NULL_PTR);
  CHECK(fastrl_token_logprob(reinterpret_cast<void*>(uintptr_t(258)), nullptr, dummy(),
                             FASTRL_BF16, 4, 64, 100, (int32_t*)dummy(), (float*)dummy(),
                             nullptr, nullptr, dummy(), 1 << 20, nullptr) == FASTRL_ERR_VALUE);
  const size_t need = fastrl_token_logprob_workspace_size(4, 64, 100, FASTRL_BF16);
  CHECK(need > 0);
  CHECK(fastrl_token_logprob(dummy(), nullptr, dummy(), FASTRL_BF16, 4, 64, 100,
                             (int32_t*)dummy(), (float*)dummy(), nullptr, nullptr, dummy(),
                             need - 1, nullptr) == FASTRL_ERR_WORKSPACE);
  CHECK(fastrl_token_logprob_noalloc(dummy(), nullptr, dummy(), FASTRL_BF16, 10, 64, 9000000,
                                     (int32_t*)dummy(), (float*)dummy(), nullptr, nullptr,
                                     nullptr) == FASTRL_ERR_SHAPE);
  CHECK(fastrl_token_logprob_noalloc_max_chunk(152064) >= 256);
  CHECK(fastrl_token_logprob_noalloc_max_chunk(9000000) == 0);
  // AdamW: bad hyper-parameters
  CHECK(fastrl_adamw_step((float*)dummy(), nullptr, (float*)dummy(), (float*)dummy(),
                          (float*)dummy(), 16, 0, 1e-6f, 0.9f, 0.999f, 1e-8f, 0.01f, 1.0f,
                          nullptr, nullptr) != FASTRL_OK);
  CHECK(fastrl_adamw_step((float*)dummy(), nullptr, (float*)dummy(), (float*)dummy(),
                          (float*)dummy(), 16, 1, 1e-6f, 1.5f, 0.999f, 1e-8f, 0.01f, 1.0f,
                          nullptr, nullptr) == FASTRL_ERR_VALUE);
}

static fastrl_loss_args loss_args(const std::vector<int64_t>& off, int64_t slab) {
  fastrl_loss_args a;
  std::memset(&a, 0, sizeof(a));
  a.hidden = a.W = dummy();
  a.token_ids = (const int32_t*)dummy();
  a.old_logp = (const float*)dummy();
  a.seq_off = (const int64_t*)dummy();
  a.adv = (const float*)dummy();
  a.loss = (float*)dummy();
  a.dtype = FASTRL_BF16;
  a.d = 3584;
  a.V = 152064;
  a.S = int32_t(off.size()) - 1;
  a.T = off.back();
  a.seq_off_host = off.data();
  a.eps_low = a.eps_high = 0.2f;
  a.slab_tokens = slab;
  return a;
}

static void slab_plans() {
  std::mt19937_64 rng(12345);
  for (int it = 0; it < 400; ++it) {
    const int S = int(rng() % 600);
    const int64_t lmax = 1 + int64_t(rng() % 20000);
    std::vector<int64_t> off(size_t(S) + 1, 0);
    int64_t longest = 0;
    for (int i = 0; i < S; ++i) {
      int64_t L = (rng() % 10 == 0) ? 0 : int64_t(rng() % uint64_t(lmax));
      longest = std::max(longest, L);
      off[size_t(i) + 1] = off[size_t(i)] + L;
    }
    const int64_t caps[] = {0, 1, 255, 4096, 32768};
    for (int64_t cap : caps) {
      fastrl_loss_args a = loss_args(off, cap);
      int64_t tc = -1;
      const int n = fastrl_policy_loss_slab_plan(&a, nullptr, 0, &tc);
      CHECK(n >= 0);
      if (n < 0) continue;
      std::vector<int32_t> begin(size_t(n) + 1, -1);
      CHECK(fastrl_policy_loss_slab_plan(&a, begin.data(), n + 1, nullptr) == n);
      const int64_t c = cap > 0 ? cap : 32768;
      CHECK(S == 0 ? n == 0 : (begin[0] == 0 && begin[size_t(n)] == S));
      int64_t mx = 0;
      for (int k = 0; k < n; ++k) {
        CHECK(begin[size_t(k) + 1] > begin[size_t(k)]);
        const int64_t tokens = off[size_t(begin[size_t(k) + 1])] - off[size_t(begin[size_t(k)])];
        CHECK(off.back() == 0 || tokens > 0);
        mx = std::max(mx, tokens);
      }
      CHECK(mx == tc);
      CHECK(tc <= std::max(c + c / 4, longest));
      CHECK(fastrl_policy_loss_workspace_size(&a) > 0);
    }
  }
  // invalid offsets are refused before any planning
  std::vector<int64_t> bad = {0, 5, 3, 9};
  fastrl_loss_args a = loss_args(bad, 0);
  CHECK(fastrl_policy_loss_slab_plan(&a, nullptr, 0, nullptr) == FASTRL_ERR_SHAPE);
  a = loss_args({0, 4, 9}, -5);
  CHECK(fastrl_policy_loss_slab_plan(&a, nullptr, 0, nullptr) == FASTRL_ERR_VALUE);
  CHECK(fastrl_loss_args_size() == sizeof(fastrl_loss_args));
}

static void ars() {
  fastrl_ars_state st;
  CHECK(fastrl_ars_init(&st, 1, 10, 2) == FASTRL_ERR_VALUE);
  CHECK(fastrl_ars_init(nullptr, 8, 10, 2) == FASTRL_ERR_NULL_PTR);
  std::mt19937_64 rng(7);
  for (int it = 0; it < 200; ++it) {
    const int G = 2 + int(rng() % 30);
    CHECK(fastrl_ars_init(&st, G, 1 + int64_t(rng() % 100), 1 + int64_t(rng() % 7)) == FASTRL_OK);
    for (int step = 0; step < 60; ++step) {
      const int Q = int(rng() % 40);
      std::vector<int32_t> cnt(size_t(Q) + 1);
      std::vector<uint8_t> valid(size_t(Q) + 1);
      for (int q = 0; q < Q; ++q) {
        cnt[size_t(q)] = 1 + int32_t(rng() % uint64_t(G));
        valid[size_t(q)] = uint8_t(rng() % 5 != 0);
      }
      CHECK(fastrl_ars_observe(&st, cnt.data(), (rng() & 1) ? valid.data() : nullptr, Q) ==
            FASTRL_OK);
      const int32_t n = fastrl_ars_next_n(&st);
      CHECK(n >= 2 && n <= G);
    }
    fastrl_ars_state copy = st;  // plain data: a copy continues identically
    const int32_t c0[3] = {1, 2, 3};
    CHECK(fastrl_ars_observe(&st, c0, nullptr, 3) == FASTRL_OK);
    CHECK(fastrl_ars_observe(&copy, c0, nullptr, 3) == FASTRL_OK);
    CHECK(std::memcmp(&st, &copy, sizeof(st)) == 0);
  }
}

int main() {
  validation_paths();
  slab_plans();
  ars();
  if (g_fail) {
    std::fprintf(stderr, "%d checks failed\n", g_fail);
    return 1;
  }
  std::printf("HOST_SANITIZE_OK\n");
  return 0;
}
