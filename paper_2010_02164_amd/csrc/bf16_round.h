// Rounding of fp64 results to bfloat16 shared by the bf16 kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace sb {

// Round a binary64 value to bfloat16 (nearest, ties to even) directly, with
// no float intermediate: keep 8 significant bits; below bf16's smallest
// normal (2^-126) the step is the subnormal quantum 2^-133.
__device__ __forceinline__ uint16_t bf16_rne_from_double(double x) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(x);
  const unsigned long long sign = u & 0x8000000000000000ull;
  unsigned long long a = u & 0x7FFFFFFFFFFFFFFFull;
  const int e = (int)(a >> 52);
  float f;
  if (e >= 1023 - 126) {
    const unsigned long long lsb = (a >> 45) & 1ull;
    a += 0x0FFFFFFFFFFFull + lsb;   // half of the dropped 45 bits, minus one
    a &= ~0x1FFFFFFFFFFFull;
    f = (float)__longlong_as_double((long long)(a | sign));
  } else {
    const double q = 0x1p-133;
    f = (float)(rint(x / q) * q);
  }
  return (uint16_t)(__float_as_uint(f) >> 16);
}

// bf16 of tanh(x) (nearest, ties to even) as if tanh were taken in fp64.
// tanh is first taken in fp32: that value is within a few fp32 ulps of the
// exact one (rounding x to fp32 adds at most one ulp, as
// |x tanh'(x)| <= |tanh(x)|), so unless it lies within 64 ulps of a tie
// between two bf16 values it rounds to the same bf16 as the exact value.
// Near a tie, and for |x| < 2^-100, tanh is taken in fp64.
__device__ __forceinline__ uint16_t bf16_tanh(double x) {
  if (fabs(x) >= 0x1p-100) {
    const uint32_t u = __float_as_uint(tanhf((float)x));
    const uint32_t lo = u & 0xFFFFu;
    if (lo < 0x8000u - 64u || lo > 0x8000u + 64u) return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
  }
  return bf16_rne_from_double(tanh(x));
}

}  // namespace sb
