// Exhaustive device check of the group-scale arithmetic of the scaled formats
// (test infrastructure): for every fp32 maximum m in [2^-112, FLT_MAX] and each
// qmax (448, 127, 7), group_scale<F>(m) must equal the correctly rounded quotient
// m / qmax (before the flush of scales below 2^-126), and for every fp32 s in
// [2^-126, 2^126) recip_scale(s) must equal the correctly rounded 1 / s. The
// references are the device's IEEE division (built with correctly rounded fp32
// division). Prints the number of values checked and of mismatches per function.
#include <hip/hip_runtime.h>

#include <cstdio>

#include "ssmq_device.hpp"

using namespace ssmq;

template <int F>
__global__ void k_check_scale(unsigned long long* bad, unsigned long long* count) {
  // bit patterns of [2^-112, FLT_MAX]: biased exponents 15 .. 254, all mantissas
  const uint32_t lo = 15u << 23, hi = 255u << 23;
  unsigned long long b = 0, n = 0;
  for (uint32_t u = lo + blockIdx.x * blockDim.x + threadIdx.x; u < hi; u += gridDim.x * blockDim.x) {
    const float m = __uint_as_float(u);
    float want = m / Traits<F>::qmax;
    if (!(want >= 1.17549435e-38f)) want = 0.0f;  // the same flush as group_scale
    b += (__float_as_uint(group_scale<F>(m)) != __float_as_uint(want));
    ++n;
  }
  atomicAdd(bad, b);
  atomicAdd(count, n);
}

__global__ void k_check_recip(unsigned long long* bad, unsigned long long* count) {
  // bit patterns of [2^-126, 2^126)
  const uint32_t lo = 1u << 23, hi = 253u << 23;
  unsigned long long b = 0, n = 0;
  for (uint32_t u = lo + blockIdx.x * blockDim.x + threadIdx.x; u < hi; u += gridDim.x * blockDim.x) {
    const float s = __uint_as_float(u);
    b += (__float_as_uint(recip_scale(s)) != __float_as_uint(1.0f / s));
    ++n;
  }
  atomicAdd(bad, b);
  atomicAdd(count, n);
}

#define CK(e) do { hipError_t r_ = (e); if (r_ != hipSuccess) { printf("HIP error %s\n", hipGetErrorString(r_)); return 1; } } while (0)

int main() {
  unsigned long long* d;
  CK(hipMalloc(&d, 8 * sizeof(unsigned long long)));
  CK(hipMemset(d, 0, 8 * sizeof(unsigned long long)));
  const dim3 grid(256 * 64), block(256);
  hipLaunchKernelGGL((k_check_scale<kE4M3>), grid, block, 0, 0, d + 0, d + 1);
  hipLaunchKernelGGL((k_check_scale<kINT8>), grid, block, 0, 0, d + 2, d + 3);
  hipLaunchKernelGGL((k_check_scale<kINT4>), grid, block, 0, 0, d + 4, d + 5);
  hipLaunchKernelGGL(k_check_recip, grid, block, 0, 0, d + 6, d + 7);
  CK(hipGetLastError());
  CK(hipDeviceSynchronize());
  unsigned long long h[8];
  CK(hipMemcpy(h, d, sizeof h, hipMemcpyDeviceToHost));
  CK(hipFree(d));
  printf("scale_e4m3 %llu %llu\nscale_int8 %llu %llu\nscale_int4 %llu %llu\nrecip %llu %llu\n",
         h[1], h[0], h[3], h[2], h[5], h[4], h[7], h[6]);
  return (h[0] | h[2] | h[4] | h[6]) ? 1 : 0;
}
