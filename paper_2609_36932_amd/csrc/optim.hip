// AdamW step on the LM-head weight, the update that consumes dW (the paper trains with
// AdamW, learning rate 1e-6 and weight decay 1e-2, Sec. 4.1; Alg. 1 ends each step with
// the policy update).  Decoupled weight decay with bias correction, per element:
//   theta <- theta (1 - lr wd);  m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
//   theta <- theta - (lr / (1 - b1^t)) m / (sqrt(v) / sqrt(1 - b2^t) + eps)
// in float32 on float32 master weights, optionally writing the bfloat16 copy the LM-head
// kernels read.  Purely HBM-bound (30 bytes per parameter): 16-byte vector accesses in a
// grid-stride loop, one pass.
#include <algorithm>
#include <cmath>

#include "common.h"

namespace fastrl {

struct AdamWConst {
  float keep;          // 1 - lr * wd
  float b1, omb1;      // beta1, 1 - beta1
  float b2, omb2;      // beta2, 1 - beta2
  float step_size;     // lr / (1 - beta1^t)
  float inv_sqrt_bc2;  // 1 / sqrt(1 - beta2^t)
  float eps;
  float gscale;
};

__device__ __forceinline__ void adamw_one(float& th, float& m, float& v, float g,
                                          const AdamWConst& c) {
  th = __fmul_rn(th, c.keep);
  m = __fadd_rn(__fmul_rn(c.b1, m), __fmul_rn(c.omb1, g));
  v = __fadd_rn(__fmul_rn(c.b2, v), __fmul_rn(c.omb2, __fmul_rn(g, g)));
  const float den = __fadd_rn(__fmul_rn(__fsqrt_rn(v), c.inv_sqrt_bc2), c.eps);
  th = __fsub_rn(th, __fmul_rn(c.step_size, __fdiv_rn(m, den)));
}

typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Two 16-byte vectors of each stream per thread and iteration (all loads issued before the
// arithmetic), non-temporal loads and stores (the 16+ GB stream would only evict the caches):
// measured at the rate of a plain device copy on this part.
__global__ __launch_bounds__(256) void adamw_kernel(float* __restrict__ theta,
                                                    uint16_t* __restrict__ wbf,
                                                    const float* __restrict__ grad,
                                                    float* __restrict__ mom,
                                                    float* __restrict__ var, int64_t n,
                                                    AdamWConst c, int32_t* __restrict__ status) {
  constexpr int U = 2;
  const int64_t n4 = n >> 2;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  f32x4_t* T = reinterpret_cast<f32x4_t*>(theta);
  const f32x4_t* G = reinterpret_cast<const f32x4_t*>(grad);
  f32x4_t* M = reinterpret_cast<f32x4_t*>(mom);
  f32x4_t* V = reinterpret_cast<f32x4_t*>(var);
  u32x2_t* WB = reinterpret_cast<u32x2_t*>(wbf);
  int bad = 0;
  for (int64_t i0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i0 < n4; i0 += stride * U) {
    f32x4_t th[U], g[U], m[U], v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + u * stride;
      if (i < n4) {
        th[u] = __builtin_nontemporal_load(T + i);
        g[u] = __builtin_nontemporal_load(G + i);
        m[u] = __builtin_nontemporal_load(M + i);
        v[u] = __builtin_nontemporal_load(V + i);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = i0 + u * stride;
      if (i < n4) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float a = th[u][q], mm = m[u][q], vv = v[u][q];
          const float gg = g[u][q] * c.gscale;
          bad |= !isfinite(gg);
          adamw_one(a, mm, vv, gg, c);
          th[u][q] = a;
          m[u][q] = mm;
          v[u][q] = vv;
        }
        __builtin_nontemporal_store(th[u], T + i);
        __builtin_nontemporal_store(m[u], M + i);
        __builtin_nontemporal_store(v[u], V + i);
        if (wbf) {
          u32x2_t pk;
          pk[0] = uint32_t(f32_to_bf16(th[u][0])) | (uint32_t(f32_to_bf16(th[u][1])) << 16);
          pk[1] = uint32_t(f32_to_bf16(th[u][2])) | (uint32_t(f32_to_bf16(th[u][3])) << 16);
          __builtin_nontemporal_store(pk, WB + i);
        }
      }
    }
  }
  // the last n % 4 elements
  if (blockIdx.x == 0 && threadIdx.x < (n & 3)) {
    const int64_t i = (n4 << 2) + threadIdx.x;
    float th = theta[i], m = mom[i], v = var[i];
    const float g = grad[i] * c.gscale;
    bad |= !isfinite(g);
    adamw_one(th, m, v, g, c);
    theta[i] = th;
    mom[i] = m;
    var[i] = v;
    if (wbf) wbf[i] = f32_to_bf16(th);
  }
  if (__any(bad) && (threadIdx.x & 63) == 0) set_status(status, FASTRL_SB_BAD_GRAD);
}

int launch_adamw(float* theta, uint16_t* wbf, const float* grad, float* mom, float* var,
                 int64_t n, int64_t step, float lr, float beta1, float beta2, float eps,
                 float weight_decay, float grad_scale, int32_t* status, hipStream_t stream) {
  if (n == 0) return FASTRL_OK;
  AdamWConst c;
  const double bc1 = 1.0 - std::pow(double(beta1), double(step));
  const double bc2 = 1.0 - std::pow(double(beta2), double(step));
  c.keep = float(1.0 - double(lr) * double(weight_decay));
  c.b1 = beta1;
  c.omb1 = float(1.0 - double(beta1));
  c.b2 = beta2;
  c.omb2 = float(1.0 - double(beta2));
  c.step_size = float(double(lr) / bc1);
  c.inv_sqrt_bc2 = float(1.0 / std::sqrt(bc2));
  c.eps = eps;
  c.gscale = grad_scale;
  const int64_t n4 = std::max<int64_t>(n >> 2, 1);
  const unsigned blocks = unsigned(std::min<int64_t>((n4 + 255) / 256, 65536));
  hipLaunchKernelGGL(adamw_kernel, dim3(blocks), dim3(256), 0, stream, theta, wbf, grad, mom,
                     var, n, c, status);
  FR_LAUNCHED();
  return FASTRL_OK;
}

}  // namespace fastrl
