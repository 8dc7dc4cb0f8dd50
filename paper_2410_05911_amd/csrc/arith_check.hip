// Device arithmetic self-check: the kernels compute three quantities with gfx950 instructions
// whose results the oracle states in plain IEEE terms.  These kernels compare the two over every
// fp32 operand of the ranges the kernels use and count the operands where they differ.
#include <hip/hip_runtime.h>

#include "../../include/aecct.h"
#include "device_common.h"

namespace aecct {
namespace {

// x in [-126, 129] (the clamped softmax argument and its neighbourhood): v_fract_f32 against
// min(x - floor(x), 1 - 2^-24), v_cvt_flr_i32_f32 against (int) floor(x), as softmax_exp2 uses them.
__global__ __launch_bounds__(256) void k_check_fract(unsigned long long *bad) {
  const uint64_t n = 2ull * 0x43010001ull;   // [+0, 129] and [-0, -126] by bit pattern
  unsigned long long cnt = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (uint64_t)gridDim.x * blockDim.x) {
    const uint32_t b = i < 0x43010001ull ? (uint32_t)i : 0x80000000u + (uint32_t)(i - 0x43010001ull);
    if (b > 0xC2FC0000u) continue;            // below -126
    const float x = __builtin_bit_cast(float, b);
    const float fr = __builtin_amdgcn_fractf(x);
    int k;
    asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(k) : "v"(x));
    float fl = __builtin_floorf(x);
    asm volatile("" : "+v"(fl));               // keeps the reference from being matched to v_fract_f32
    float d = x - fl;
    asm volatile("" : "+v"(d));
    const float ref = __builtin_fminf(d, 0x1.fffffep-1f);
    cnt += (__builtin_bit_cast(uint32_t, fr) != __builtin_bit_cast(uint32_t, ref)) | (k != (int)fl);
  }
  if (cnt) atomicAdd(bad, cnt);
}

// s in [2^-64, 2^64]: recip_softmax_sum(s) against the IEEE quotient 1 / s.
__global__ __launch_bounds__(256) void k_check_recip(unsigned long long *bad) {
  const uint32_t lo = 0x1F800000u, count = 0x5F800000u - 0x1F800000u + 1u;
  unsigned long long cnt = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (uint64_t)gridDim.x * blockDim.x) {
    const float s = __builtin_bit_cast(float, lo + (uint32_t)i);
    cnt += __builtin_bit_cast(uint32_t, recip_softmax_sum(s)) != __builtin_bit_cast(uint32_t, 1.0f / s);
  }
  if (cnt) atomicAdd(bad, cnt);
}

// every finite fp32 a >= 0 (zero, denormals, normals): inv127(a) against a == 0 ? 0 : 127 / a.
__global__ __launch_bounds__(256) void k_check_inv127(unsigned long long *bad) {
  const uint64_t count = 0x7F800000ull;
  unsigned long long cnt = 0;
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += (uint64_t)gridDim.x * blockDim.x) {
    const float a = __builtin_bit_cast(float, (uint32_t)i);
    const float ref = a == 0.0f ? 0.0f : 127.0f / a;
    cnt += __builtin_bit_cast(uint32_t, inv127(a)) != __builtin_bit_cast(uint32_t, ref);
  }
  if (cnt) atomicAdd(bad, cnt);
}

}  // namespace
}  // namespace aecct

extern "C" aecct_status aecct_check_device_arith(uint64_t *counts) {
  if (!counts) return AECCT_ERR_INVALID_ARG;
  int dev_count = 0;
  if (hipGetDeviceCount(&dev_count) != hipSuccess || dev_count < 1) return AECCT_ERR_DEVICE;
  unsigned long long *d = nullptr;
  if (hipMalloc((void **)&d, 3 * sizeof(unsigned long long)) != hipSuccess) return AECCT_ERR_DEVICE;
  hipError_t e = hipMemset(d, 0, 3 * sizeof(unsigned long long));
  if (e == hipSuccess) {
    hipLaunchKernelGGL(aecct::k_check_fract, dim3(4096), dim3(256), 0, 0, d);
    hipLaunchKernelGGL(aecct::k_check_recip, dim3(4096), dim3(256), 0, 0, d + 1);
    hipLaunchKernelGGL(aecct::k_check_inv127, dim3(4096), dim3(256), 0, 0, d + 2);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  unsigned long long h[3] = {0, 0, 0};
  if (e == hipSuccess) e = hipMemcpy(h, d, sizeof(h), hipMemcpyDeviceToHost);
  (void)hipFree(d);
  if (e != hipSuccess) return AECCT_ERR_DEVICE;
  for (int i = 0; i < 3; ++i) counts[i] = h[i];
  return AECCT_OK;
}
