// Internal helpers shared by the gfx950 kernels and the C-ABI layer.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string>

#include "../../include/fastrl.h"

namespace fastrl {

// ---- error handling -------------------------------------------------------------------
void set_error(const std::string& msg);
void clear_error();

#define FR_CHECK_ARG(cond, code, msg)  \
  do {                                 \
    if (!(cond)) {                     \
      ::fastrl::set_error(msg);        \
      return (code);                   \
    }                                  \
  } while (0)

#define FR_HIP(call)                                                              \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess) {                                                       \
      ::fastrl::set_error(std::string(#call) + ": " + hipGetErrorString(e_));     \
      return FASTRL_ERR_HIP;                                                      \
    }                                                                             \
  } while (0)

// launch-error check (kernel launch configuration errors are reported here)
#define FR_LAUNCHED() FR_HIP(hipGetLastError())

// ---- workspace carving ----------------------------------------------------------------
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t size() const { return (off + 255) & ~size_t(255); }
};

// ---- bf16 helpers ----------------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float(uint32_t(h) << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {  // round to nearest even
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ void set_status(int32_t* status, int32_t bit) {
  if (status) atomicOr(status, bit);
}

// kernel timing recorder (fastrl_profile_*)
struct ProfScope {
  int kind;
  hipStream_t stream;
  double flops;
  void* ev0 = nullptr;
  ProfScope(int k, hipStream_t s, double f);
  ~ProfScope();
};

}  // namespace fastrl
