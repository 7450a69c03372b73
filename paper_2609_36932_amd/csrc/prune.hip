// Maximizing Differential Advantage Pruning (Sec. 3.2; Alg. 1 Phase 2), the keep-ratio
// budget, and stream compaction of kept tokens.  Every decision is integer or exact:
//   K1 ngram_sort   one block per trajectory: pack n-grams into 64-bit keys (21 bits per
//                   token), bitonic-sort them in LDS, keep the distinct ones.
//   K2 pair_conflict one block per question: |N_n(o_i) & N_n(o_j)| for every same-class
//                   pair by binary search of the shorter key list in the longer one, then
//                   theta < tau as  tau_den * (|U| - |I|) < tau_num * |U|  in int64.
//   K0 group_eps    (continuous rewards, appendix on the grounding task) one wavefront per
//                   question: classes = connected components of |A_i - A_j| < eps, from the
//                   sorted advantages (a new class wherever a gap is >= eps).
//   K3 select       one wavefront per question: the greedy independent set in visiting
//                   order (|A| descending, ties by index, when advantages are given; else
//                   ascending index), then the budget as "keep the K smallest (tier, rank,
//                   class position) keys" -- the same list a class round-robin produces.
//   K3b dp_fill     (optional) Alg. 1's DP alignment of the kept count, one block.
//   K4 compaction   exclusive scans of kept flags and kept lengths (one block), then a
//                   coalesced fill of tok_src, one block per kept trajectory.
#include "common.h"

namespace fastrl {

constexpr int kMaxGroupPrune = 256;
constexpr int kMaxLenPrune = 16384;
constexpr uint64_t kKeyPad = ~0ull;

// ---------------------------------------------------------------------------- K1
__global__ __launch_bounds__(256) void ngram_sort_kernel(
    const int32_t* __restrict__ tokens, const int64_t* __restrict__ toff, int64_t T_total,
    int32_t N, int32_t V, int32_t n, int32_t max_len, int32_t P, uint64_t* __restrict__ keys,
    int32_t* __restrict__ nuniq, int32_t* __restrict__ status) {
  extern __shared__ uint64_t sk[];  // P keys, then P/ (reused) int32 scan area follows
  __shared__ int32_t wsum[4];
  __shared__ int32_t bad_flag;
  const int i = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t a = toff[i], b = toff[i + 1];
  if (tid == 0) bad_flag = 0;
  __syncthreads();
  if (a < 0 || b < a || b > T_total) {
    if (tid == 0) {
      set_status(status, FASTRL_SB_BAD_OFFSETS);
      nuniq[i] = 0;
    }
    return;
  }
  const int64_t L = b - a;
  if (L > max_len) {
    if (tid == 0) {
      set_status(status, FASTRL_SB_SEQ_TOO_LONG);
      nuniq[i] = 0;
    }
    return;
  }
  const int m = L >= n ? int(L - n + 1) : 0;
  for (int j = tid; j < P; j += 256) {
    uint64_t key = kKeyPad;
    if (j < m) {
      key = 0;
      for (int k = 0; k < n; ++k) {
        int32_t t = tokens[a + j + k];
        if (t < 0 || t >= V) {
          bad_flag = 1;
          t = 0;
        }
        key |= uint64_t(uint32_t(t)) << (21 * k);
      }
    }
    sk[j] = key;
  }
  __syncthreads();
  if (bad_flag && tid == 0) set_status(status, FASTRL_SB_BAD_TOKEN);
  // bitonic sort, ascending
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int j = tid; j < (P >> 1); j += 256) {
        const int lo = 2 * j - (j & (stride - 1));
        const int hi = lo + stride;
        const bool up = ((lo & size) == 0);
        const uint64_t x = sk[lo], y = sk[hi];
        if ((x > y) == up) {
          sk[lo] = y;
          sk[hi] = x;
        }
      }
      __syncthreads();
    }
  }
  // distinct keys, written in order: block-wide exclusive scan over chunks of 256
  int base = 0;
  const int lane = tid & 63, wv = tid >> 6;
  for (int c = 0; c < m; c += 256) {
    const int j = c + tid;
    const int f = (j < m) && (j == 0 || sk[j] != sk[j - 1]);
    // wave inclusive scan
    int v = f;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int t = __shfl_up(v, o, 64);
      if (lane >= o) v += t;
    }
    if (lane == 63) wsum[wv] = v;
    __syncthreads();
    int pre = 0, tot = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wv) pre += wsum[w];
      tot += wsum[w];
    }
    if (f) keys[a + base + pre + v - 1] = sk[j];
    base += tot;
    __syncthreads();
  }
  if (tid == 0) nuniq[i] = base;
}

// ---------------------------------------------------------------------------- K0
// Continuous-reward classes of one question: the connected components of the relation
// |A_i - A_j| < eps over its float32 advantages (read as float64, gaps in float64),
// numbered by lowest member index.  Sorting by (A, index) puts every component on a run of
// consecutive positions, and a run ends where the gap to the next value is >= eps.
__global__ __launch_bounds__(64) void group_eps_kernel(
    const float* __restrict__ adv, const int32_t* __restrict__ group_off, int32_t N,
    int32_t max_group, double eps, int32_t* __restrict__ cls_out, int32_t* __restrict__ status) {
  __shared__ float a[kMaxGroupPrune];
  __shared__ int32_t sidx[kMaxGroupPrune];   // position -> member
  __shared__ int32_t comp[kMaxGroupPrune];   // member -> component (in sorted order)
  __shared__ int32_t label[kMaxGroupPrune];  // component -> class id
  const int q = blockIdx.x;
  const int lane = threadIdx.x;
  const int g0 = group_off[q], g1 = group_off[q + 1];
  if (g0 < 0 || g1 < g0 || g1 > N || g1 - g0 > max_group) return;  // flagged by K3
  const int G = g1 - g0;
  int bad = 0;
  for (int i = lane; i < G; i += 64) {
    float v = adv[g0 + i];
    if (!isfinite(v)) {  // keeps the ranks a permutation
      bad = 1;
      v = 0.0f;
    }
    a[i] = v;
  }
  if (bad) set_status(status, FASTRL_SB_BAD_REWARD);
  __syncthreads();
  for (int i = lane; i < G; i += 64) {
    const float ai = a[i];
    int r = 0;
    for (int j = 0; j < G; ++j) r += (a[j] < ai) || (a[j] == ai && j < i);
    sidx[r] = i;
  }
  __syncthreads();
  if (lane == 0 && G > 0) {
    int c = 0;
    comp[sidx[0]] = 0;
    for (int p = 1; p < G; ++p) {
      if (__dsub_rn(double(a[sidx[p]]), double(a[sidx[p - 1]])) >= eps) ++c;
      comp[sidx[p]] = c;
    }
    for (int k = 0; k <= c; ++k) label[k] = -1;
    int next = 0;
    for (int i = 0; i < G; ++i) {
      const int k = comp[i];
      if (label[k] < 0) label[k] = next++;
      cls_out[g0 + i] = label[k];
    }
  }
}

// ---------------------------------------------------------------------------- K2
__global__ __launch_bounds__(256) void pair_conflict_kernel(
    const int64_t* __restrict__ toff, const int32_t* __restrict__ group_off,
    const int32_t* __restrict__ class_id, const uint64_t* __restrict__ keys,
    const int32_t* __restrict__ nuniq, int32_t N, int32_t max_group, int32_t tau_num,
    int32_t tau_den, uint8_t* __restrict__ conflict) {
  const int q = blockIdx.x;
  const int g0 = group_off[q], g1 = group_off[q + 1];
  if (g0 < 0 || g1 < g0 || g1 > N || g1 - g0 > max_group) return;  // flagged by K3
  const int G = g1 - g0;
  const int npairs = G * (G - 1) / 2;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint8_t* cq = conflict + size_t(q) * max_group * max_group;
  for (int p = wv; p < npairs; p += 4) {
    // p -> (i, j), i > j:  p = i (i - 1) / 2 + j
    int i = int((1.0 + sqrt(1.0 + 8.0 * double(p))) * 0.5);
    while (i * (i - 1) / 2 > p) --i;
    while ((i + 1) * i / 2 <= p) ++i;
    const int j = p - i * (i - 1) / 2;
    if (class_id[g0 + i] != class_id[g0 + j]) continue;
    const int na = nuniq[g0 + i], nb = nuniq[g0 + j];
    const uint64_t* ka = keys + toff[g0 + i];
    const uint64_t* kb = keys + toff[g0 + j];
    const uint64_t* ks = na <= nb ? ka : kb;  // shorter list, searched in the longer
    const uint64_t* kl = na <= nb ? kb : ka;
    const int ns = na <= nb ? na : nb, nl = na <= nb ? nb : na;
    int cnt = 0;
    for (int e = lane; e < ns; e += 64) {
      const uint64_t x = ks[e];
      int lo = 0, hi = nl;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        if (kl[mid] < x) lo = mid + 1; else hi = mid;
      }
      cnt += (lo < nl && kl[lo] == x);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
    if (lane == 0) {
      const int64_t I = cnt, U = int64_t(na) + nb - cnt;
      bool c;
      if (U == 0) c = tau_num > 0;  // theta = 0 for two empty sets
      else c = int64_t(tau_den) * (U - I) < int64_t(tau_num) * U;
      cq[i * max_group + j] = c;
      cq[j * max_group + i] = c;
    }
  }
}

// ---------------------------------------------------------------------------- K3
__global__ __launch_bounds__(64) void select_kernel(
    const float* __restrict__ rewards, const int32_t* __restrict__ group_off,
    const int32_t* __restrict__ class_id, const float* __restrict__ adv,
    const uint8_t* __restrict__ group_valid, int32_t N, int32_t max_group, double keep_ratio,
    const uint8_t* __restrict__ conflict, uint8_t* __restrict__ keep_mask,
    int32_t* __restrict__ mdap_count, int32_t* __restrict__ class_out,
    int32_t* __restrict__ status) {
  __shared__ uint8_t mdap[kMaxGroupPrune];
  __shared__ int32_t cls[kMaxGroupPrune];
  __shared__ int32_t vpos[kMaxGroupPrune];     // visiting position of member i
  __shared__ int32_t ord[kMaxGroupPrune];      // member at visiting position p
  __shared__ float aabs[kMaxGroupPrune];
  __shared__ int32_t crep[kMaxGroupPrune];     // first visited member of class c
  __shared__ int32_t cmin[kMaxGroupPrune];     // lowest member index of class c
  __shared__ double kappa[kMaxGroupPrune];     // kappa of class c
  __shared__ int32_t cpos[kMaxGroupPrune];     // rank of class c in the budget order
  __shared__ int32_t rank[kMaxGroupPrune];     // rank of member i inside its class tier
  const int q = blockIdx.x;
  const int lane = threadIdx.x;
  const int g0 = group_off[q], g1 = group_off[q + 1];
  if (g0 < 0 || g1 < g0 || g1 > N) {
    if (lane == 0) {
      set_status(status, FASTRL_SB_BAD_OFFSETS);
      mdap_count[q] = 0;
    }
    return;
  }
  const int G = g1 - g0;
  if (G > max_group) {
    for (int i = lane; i < G; i += 64) keep_mask[g0 + i] = 0;
    if (lane == 0) {
      set_status(status, FASTRL_SB_GROUP_TOO_BIG);
      mdap_count[q] = 0;
    }
    return;
  }
  for (int i = lane; i < G; i += 64) {
    int c = class_id[g0 + i];
    if (c < 0 || c >= G) {  // class ids are 0..G-1
      set_status(status, FASTRL_SB_BAD_INDEX);
      c = 0;
    }
    cls[i] = c;
    if (class_out) class_out[g0 + i] = c;
  }
  const bool valid = group_valid ? group_valid[q] != 0 : true;
  if (!valid || G == 0) {
    for (int i = lane; i < G; i += 64) keep_mask[g0 + i] = 0;
    if (lane == 0) mdap_count[q] = 0;
    return;
  }
  // visiting order: |A| descending, ties by index (Alg. 1); ascending index without A
  if (adv) {
    for (int i = lane; i < G; i += 64) {
      const float v = adv[g0 + i];
      aabs[i] = isfinite(v) ? fabsf(v) : 0.0f;  // non-finite A was flagged upstream
    }
    __syncthreads();
    for (int i = lane; i < G; i += 64) {
      const float ai = aabs[i];
      int r = 0;
      for (int j = 0; j < G; ++j) r += (aabs[j] > ai) || (aabs[j] == ai && j < i);
      vpos[i] = r;
      ord[r] = i;
    }
  } else {
    for (int i = lane; i < G; i += 64) {
      vpos[i] = i;
      ord[i] = i;
    }
  }
  __syncthreads();
  const uint8_t* cq = conflict + size_t(q) * max_group * max_group;
  if (lane == 0) {
    // greedy maximal independent set per class, members in visiting order
    int count = 0;
    for (int p = 0; p < G; ++p) {
      const int i = ord[p];
      uint8_t keep = 1;
      for (int pj = 0; pj < p; ++pj) {
        const int j = ord[pj];
        if (mdap[j] && cls[j] == cls[i] && cq[i * max_group + j]) {
          keep = 0;
          break;
        }
      }
      mdap[i] = keep;
      count += keep;
    }
    mdap_count[q] = count;
  }
  __syncthreads();
  if (!(keep_ratio > 0.0)) {
    for (int i = lane; i < G; i += 64) keep_mask[g0 + i] = mdap[i];
    return;
  }
  // budget: kappa_k = |G r_k - sum_j r_j| (sum in index order, float64; r_k the reward of
  // the class's first visited member); classes ordered by kappa descending, then by their
  // lowest member index
  for (int c = lane; c < G; c += 64) {
    crep[c] = -1;
    cmin[c] = -1;
  }
  __syncthreads();
  if (lane == 0) {
    double s = 0.0;
    for (int j = 0; j < G; ++j) s = __dadd_rn(s, double(rewards[g0 + j]));
    for (int p = 0; p < G; ++p) {
      const int j = ord[p];
      const int c = cls[j];
      if (crep[c] < 0) {
        crep[c] = j;
        kappa[c] = fabs(__dsub_rn(__dmul_rn(double(G), double(rewards[g0 + j])), s));
      }
    }
    for (int j = 0; j < G; ++j)
      if (cmin[cls[j]] < 0) cmin[cls[j]] = j;
  }
  __syncthreads();
  for (int c = lane; c < G; c += 64) {
    if (crep[c] < 0) continue;
    int pos = 0;
    for (int e = 0; e < G; ++e) {
      if (crep[e] < 0 || e == c) continue;
      if (kappa[e] > kappa[c] || (kappa[e] == kappa[c] && cmin[e] < cmin[c])) ++pos;
    }
    cpos[c] = pos;
  }
  __syncthreads();
  const double kf = floor(__dadd_rn(__dmul_rn(keep_ratio, double(G)), 0.5));
  const int K = kf < 1.0 ? 1 : (kf > double(G) ? G : int(kf));
  for (int i = lane; i < G; i += 64) {
    const int ti = mdap[i] ? 0 : 1;
    int ri = 0;
    for (int j = 0; j < G; ++j)
      ri += (cls[j] == cls[i] && (mdap[j] ? 0 : 1) == ti && vpos[j] < vpos[i]);
    rank[i] = ri;
  }
  __syncthreads();
  for (int i = lane; i < G; i += 64) {
    // key(i) = (tier, rank within class tier, class position); keep the K smallest
    const int ti = mdap[i] ? 0 : 1, ri = rank[i], pi = cpos[cls[i]];
    int smaller = 0;
    for (int j = 0; j < G; ++j) {
      const int tj = mdap[j] ? 0 : 1, rj = rank[j], pj = cpos[cls[j]];
      smaller += (tj != ti) ? (tj < ti) : (rj != ri ? rj < ri : pj < pi);
    }
    keep_mask[g0 + i] = smaller < K ? 1 : 0;
  }
}

// ---------------------------------------------------------------------------- K3b
// DP alignment (Alg. 1 after the union of the per-question sets): while the kept count is
// not a multiple of d, add the unselected trajectory with the highest |A|, round-robin over
// the questions.  One block: count the kept set; rank every unselected member of a valid
// question by (|A| descending, index); one thread deals the rounds to get t_q, the number of
// members question q contributes; members of rank < t_q are kept.
__global__ __launch_bounds__(1024) void dp_fill_kernel(
    uint8_t* __restrict__ keep_mask, const float* __restrict__ adv,
    const int32_t* __restrict__ group_off, const uint8_t* __restrict__ group_valid, int32_t Q,
    int32_t N, int32_t max_group, int32_t d, int32_t* __restrict__ frank,
    int32_t* __restrict__ unsel, int32_t* __restrict__ take, int32_t* __restrict__ status) {
  __shared__ int32_t red[16];
  __shared__ int32_t need_s;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int c = 0;
  for (int i = tid; i < N; i += blockDim.x) c += keep_mask[i] ? 1 : 0;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o, 64);
  if (lane == 0) red[wv] = c;
  __syncthreads();
  if (tid == 0) {
    int kept = 0;
    for (int w = 0; w < int(blockDim.x >> 6); ++w) kept += red[w];
    need_s = (d - kept % d) % d;
  }
  __syncthreads();
  if (need_s == 0) return;
  for (int q = tid; q < Q; q += blockDim.x) {
    const int g0 = group_off[q], g1 = group_off[q + 1];
    int u = 0;
    const bool ok = g0 >= 0 && g1 >= g0 && g1 <= N && g1 - g0 <= max_group &&
                    (group_valid == nullptr || group_valid[q] != 0);
    if (ok) {
      for (int i = g0; i < g1; ++i) {
        if (keep_mask[i]) continue;
        const float ai = isfinite(adv[i]) ? fabsf(adv[i]) : 0.0f;
        int r = 0;
        for (int j = g0; j < g1; ++j) {
          if (keep_mask[j]) continue;
          const float aj = isfinite(adv[j]) ? fabsf(adv[j]) : 0.0f;
          r += (aj > ai) || (aj == ai && j < i);
        }
        frank[i] = r;
        ++u;
      }
    }
    unsel[q] = u;
    take[q] = 0;
  }
  __syncthreads();
  if (tid == 0) {
    int need = need_s;
    for (int r = 0; need > 0; ++r) {
      bool any = false;
      for (int q = 0; q < Q && need > 0; ++q) {
        if (unsel[q] > r) {
          take[q] = r + 1;
          --need;
          any = true;
        }
      }
      if (!any) break;
    }
    if (need > 0) set_status(status, FASTRL_SB_FILL_SHORT);
  }
  __syncthreads();
  for (int q = tid; q < Q; q += blockDim.x) {
    const int t = take[q];
    if (t == 0) continue;
    const int g0 = group_off[q], g1 = group_off[q + 1];
    for (int i = g0; i < g1; ++i)
      if (!keep_mask[i] && frank[i] < t) keep_mask[i] = 1;  // ranks were taken above
  }
}

// ---------------------------------------------------------------------------- K4
__global__ __launch_bounds__(1024) void compact_scan_kernel(
    const uint8_t* __restrict__ keep_mask, const int64_t* __restrict__ toff, int32_t N,
    int32_t* __restrict__ kept_traj, int64_t* __restrict__ kept_tok_off,
    int32_t* __restrict__ kpos, int64_t* __restrict__ counts) {
  __shared__ int32_t wc[16];
  __shared__ int64_t wl[16];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  int32_t base_n = 0;
  int64_t base_t = 0;
  for (int c = 0; c < N; c += 1024) {
    const int i = c + tid;
    const int f = (i < N) ? (keep_mask[i] != 0) : 0;
    const int64_t len = f ? (toff[i + 1] - toff[i]) : 0;
    int vn = f;
    int64_t vl = len;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      int tn = __shfl_up(vn, o, 64);
      int64_t tl = __shfl_up(vl, o, 64);
      if (lane >= o) {
        vn += tn;
        vl += tl;
      }
    }
    if (lane == 63) {
      wc[wv] = vn;
      wl[wv] = vl;
    }
    __syncthreads();
    int32_t pn = 0, totn = 0;
    int64_t pl = 0, totl = 0;
    for (int w = 0; w < 16; ++w) {
      if (w < wv) {
        pn += wc[w];
        pl += wl[w];
      }
      totn += wc[w];
      totl += wl[w];
    }
    if (i < N) {
      const int32_t pos = base_n + pn + vn - f;
      kpos[i] = f ? pos : -1;
      if (f) {
        kept_traj[pos] = i;
        kept_tok_off[pos] = base_t + pl + vl - len;
      }
    }
    base_n += totn;
    base_t += totl;
    __syncthreads();
  }
  if (tid == 0) {
    kept_tok_off[base_n] = base_t;
    counts[0] = base_n;
    counts[1] = base_t;
  }
}

__global__ __launch_bounds__(256) void compact_fill_kernel(
    const int32_t* __restrict__ kpos, const int64_t* __restrict__ toff,
    const int64_t* __restrict__ kept_tok_off, int32_t* __restrict__ tok_src) {
  const int i = blockIdx.x;
  const int pos = kpos[i];
  if (pos < 0) return;
  const int64_t a = toff[i], L = toff[i + 1] - a;
  const int64_t dst = kept_tok_off[pos];
  for (int64_t t = threadIdx.x; t < L; t += 256) tok_src[dst + t] = int32_t(a + t);
}

// ---------------------------------------------------------------------------- host
static int next_pow2(int x) {
  int p = 1;
  while (p < x) p <<= 1;
  return p;
}

size_t prune_workspace(int32_t Q, int32_t N, int64_t T_total, int32_t max_group) {
  Carver c(nullptr);
  c.take<uint64_t>(size_t(T_total > 0 ? T_total : 1));
  c.take<int32_t>(size_t(N + 1));
  c.take<uint8_t>(size_t(Q > 0 ? Q : 1) * max_group * max_group);
  c.take<int32_t>(size_t(N + 1));
  c.take<int32_t>(size_t(N + 1));
  c.take<int32_t>(size_t(N + 1));
  c.take<int32_t>(size_t(Q + 1));
  c.take<int32_t>(size_t(Q + 1));
  return c.size();
}

int launch_prune(const int32_t* token_ids, const int64_t* toff, int64_t T_total,
                 const float* rewards, const int32_t* group_off, const int32_t* class_id,
                 const float* adv, double group_eps, const uint8_t* group_valid, int32_t Q,
                 int32_t N, int32_t max_group, int32_t max_len, int32_t V, int32_t ngram_n,
                 int32_t tau_num, int32_t tau_den, double keep_ratio, uint8_t* keep_mask,
                 int32_t* mdap_count, int32_t* class_out, int32_t dp_align, int32_t* kept_traj,
                 int64_t* kept_tok_off, int32_t* tok_src, int64_t* counts, int32_t* status,
                 void* ws, hipStream_t stream) {
  Carver c(ws);
  uint64_t* keys = c.take<uint64_t>(size_t(T_total > 0 ? T_total : 1));
  int32_t* nuniq = c.take<int32_t>(size_t(N + 1));
  uint8_t* conflict = c.take<uint8_t>(size_t(Q > 0 ? Q : 1) * max_group * max_group);
  int32_t* kpos = c.take<int32_t>(size_t(N + 1));
  int32_t* cls_eps = c.take<int32_t>(size_t(N + 1));
  int32_t* frank = c.take<int32_t>(size_t(N + 1));
  int32_t* unsel = c.take<int32_t>(size_t(Q + 1));
  int32_t* take = c.take<int32_t>(size_t(Q + 1));
  const int32_t* cls = class_id;
  if (group_eps > 0.0 && Q > 0) {
    hipLaunchKernelGGL(group_eps_kernel, dim3(Q), dim3(64), 0, stream, adv, group_off, N,
                       max_group, group_eps, cls_eps, status);
    FR_LAUNCHED();
    cls = cls_eps;
  }
  if (N > 0) {
    const int P = next_pow2(max_len > 1 ? max_len : 1);
    const size_t shm = size_t(P) * sizeof(uint64_t);
    if (shm > 64 * 1024)
      FR_HIP(hipFuncSetAttribute((const void*)ngram_sort_kernel,
                                 hipFuncAttributeMaxDynamicSharedMemorySize, int(shm)));
    hipLaunchKernelGGL(ngram_sort_kernel, dim3(N), dim3(256), shm, stream, token_ids, toff,
                       T_total, N, V, ngram_n, max_len, P, keys, nuniq, status);
    FR_LAUNCHED();
  }
  if (Q > 0) {
    hipLaunchKernelGGL(pair_conflict_kernel, dim3(Q), dim3(256), 0, stream, toff, group_off,
                       cls, keys, nuniq, N, max_group, tau_num, tau_den, conflict);
    FR_LAUNCHED();
    hipLaunchKernelGGL(select_kernel, dim3(Q), dim3(64), 0, stream, rewards, group_off, cls,
                       adv, group_valid, N, max_group, keep_ratio, conflict, keep_mask,
                       mdap_count, class_out, status);
    FR_LAUNCHED();
    if (dp_align > 1) {
      hipLaunchKernelGGL(dp_fill_kernel, dim3(1), dim3(1024), 0, stream, keep_mask, adv,
                         group_off, group_valid, Q, N, max_group, dp_align, frank, unsel, take,
                         status);
      FR_LAUNCHED();
    }
  }
  hipLaunchKernelGGL(compact_scan_kernel, dim3(1), dim3(1024), 0, stream, keep_mask, toff, N,
                     kept_traj, kept_tok_off, kpos, counts);
  FR_LAUNCHED();
  if (N > 0) {
    hipLaunchKernelGGL(compact_fill_kernel, dim3(N), dim3(256), 0, stream, kpos, toff,
                       kept_tok_off, tok_src);
    FR_LAUNCHED();
  }
  return FASTRL_OK;
}

}  // namespace fastrl
