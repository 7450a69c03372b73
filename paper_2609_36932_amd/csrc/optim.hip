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

__global__ __launch_bounds__(256) void adamw_kernel(float* __restrict__ theta,
                                                    uint16_t* __restrict__ wbf,
                                                    const float* __restrict__ grad,
                                                    float* __restrict__ mom,
                                                    float* __restrict__ var, int64_t n,
                                                    AdamWConst c, int32_t* __restrict__ status) {
  const int64_t n4 = n >> 2;
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  int bad = 0;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 th = reinterpret_cast<const float4*>(theta)[i];
    const float4 gr = reinterpret_cast<const float4*>(grad)[i];
    float4 m = reinterpret_cast<const float4*>(mom)[i];
    float4 v = reinterpret_cast<const float4*>(var)[i];
    const float g0 = gr.x * c.gscale, g1 = gr.y * c.gscale, g2 = gr.z * c.gscale,
                g3 = gr.w * c.gscale;
    bad |= !(isfinite(g0) && isfinite(g1) && isfinite(g2) && isfinite(g3));
    adamw_one(th.x, m.x, v.x, g0, c);
    adamw_one(th.y, m.y, v.y, g1, c);
    adamw_one(th.z, m.z, v.z, g2, c);
    adamw_one(th.w, m.w, v.w, g3, c);
    reinterpret_cast<float4*>(theta)[i] = th;
    reinterpret_cast<float4*>(mom)[i] = m;
    reinterpret_cast<float4*>(var)[i] = v;
    if (wbf) {
      uint2 pk;
      pk.x = uint32_t(f32_to_bf16(th.x)) | (uint32_t(f32_to_bf16(th.y)) << 16);
      pk.y = uint32_t(f32_to_bf16(th.z)) | (uint32_t(f32_to_bf16(th.w)) << 16);
      reinterpret_cast<uint2*>(wbf)[i] = pk;
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
  const unsigned blocks = unsigned(std::min<int64_t>((n4 + 255) / 256, 256 * 8));
  hipLaunchKernelGGL(adamw_kernel, dim3(blocks), dim3(256), 0, stream, theta, wbf, grad, mom,
                     var, n, c, status);
  FR_LAUNCHED();
  return FASTRL_OK;
}

}  // namespace fastrl
