// Group-normalised advantage and advantage classes (Sec. 3.2, Eq. advantage and
// Eq. grouping).  One 64-wide wavefront per question: one lane sums the rewards in index
// order in float64 (correctly rounded operations, no contraction), then every lane writes
// its members.  The groups are small (G <= 1024), and the fixed order makes the float32
// advantages exactly reproducible, which the continuous-reward grouping of the pruning
// step relies on (its decisions compare advantages against a threshold).
#include "common.h"

namespace fastrl {

constexpr int kAdvWaves = 4;       // questions per 256-thread block
constexpr int kAdvMaxGroup = 1024;

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void advantage_kernel(
    const float* __restrict__ rewards, const int32_t* __restrict__ group_off, int32_t Q,
    int32_t N, int32_t ddof, float eps, int32_t drop_uniform, float* __restrict__ adv,
    int32_t* __restrict__ class_id, uint8_t* __restrict__ group_valid,
    int32_t* __restrict__ status) {
  __shared__ uint8_t first_flag[kAdvWaves][kAdvMaxGroup];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int q = blockIdx.x * kAdvWaves + wave;
  if (q >= Q) return;
  const int a = group_off[q];
  const int b = group_off[q + 1];
  if (a < 0 || b < a || b > N) {
    if (lane == 0) {
      set_status(status, FASTRL_SB_BAD_OFFSETS);
      group_valid[q] = 0;
    }
    return;
  }
  const int G = b - a;
  if (G > kAdvMaxGroup) {
    if (lane == 0) {
      set_status(status, FASTRL_SB_GROUP_TOO_BIG);
      group_valid[q] = 0;
    }
    return;
  }
  if (G == 0) {
    if (lane == 0) group_valid[q] = 0;
    return;
  }
  // mean and std in float64, summed in index order by one lane with explicitly rounded
  // operations (no contraction), so A is reproducible bit for bit from the rewards
  int bad = 0;
  for (int i = lane; i < G; i += 64) bad |= !isfinite(rewards[a + i]);
  if (wave_sum_i(bad) && lane == 0) set_status(status, FASTRL_SB_BAD_REWARD);
  double mean = 0.0, sd = 0.0;
  if (lane == 0) {
    double s1 = 0.0;
    for (int i = 0; i < G; ++i) s1 = __dadd_rn(s1, double(rewards[a + i]));
    mean = __ddiv_rn(s1, double(G));
    double s2 = 0.0;
    for (int i = 0; i < G; ++i) {
      const double dv = __dsub_rn(double(rewards[a + i]), mean);
      s2 = __dadd_rn(s2, __dmul_rn(dv, dv));
    }
    sd = (G - ddof > 0) ? __dsqrt_rn(__ddiv_rn(s2, double(G - ddof))) : 0.0;
  }
  mean = __shfl(mean, 0, 64);
  sd = __shfl(sd, 0, 64);
  const double den = __dadd_rn(sd, double(eps));
  // classes: first occurrence of each distinct reward value
  int nfirst = 0;
  for (int i = lane; i < G; i += 64) {
    const float r = rewards[a + i];
    int first = 1;
    for (int j = 0; j < i; ++j) {
      if (rewards[a + j] == r) {
        first = 0;
        break;
      }
    }
    first_flag[wave][i] = uint8_t(first);
    nfirst += first;
  }
  nfirst = wave_sum_i(nfirst);
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  for (int i = lane; i < G; i += 64) {
    const float r = rewards[a + i];
    int f = i;
    for (int j = 0; j < i; ++j) {
      if (rewards[a + j] == r) {
        f = j;
        break;
      }
    }
    int cls = 0;
    for (int k = 0; k < f; ++k) cls += first_flag[wave][k];
    class_id[a + i] = cls;
    const double num = __dsub_rn(double(r), mean);
    adv[a + i] = (den > 0.0) ? float(__ddiv_rn(num, den)) : 0.0f;
  }
  if (lane == 0) group_valid[q] = (drop_uniform && nfirst == 1) ? 0 : 1;
}

int launch_advantage(const float* rewards, const int32_t* group_off, int32_t Q, int32_t N,
                     int32_t ddof, float eps, int32_t drop_uniform, float* adv,
                     int32_t* class_id, uint8_t* group_valid, int32_t* status,
                     hipStream_t stream) {
  if (Q == 0) return FASTRL_OK;
  dim3 grid((Q + kAdvWaves - 1) / kAdvWaves);
  hipLaunchKernelGGL(advantage_kernel, grid, dim3(256), 0, stream, rewards, group_off, Q, N,
                     ddof, eps, drop_uniform, adv, class_id, group_valid, status);
  FR_LAUNCHED();
  return FASTRL_OK;
}

}  // namespace fastrl
