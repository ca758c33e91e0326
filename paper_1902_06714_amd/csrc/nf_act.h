// f(z) and f'(z) of the activation functions, shared by the device kernels,
// in the two precisions of the library (fp32, the paper's default real kind,
// and fp64, its real64 kind).
#pragma once

#include <hip/hip_runtime.h>

namespace nf {

enum { ACT_GAUSSIAN = 0, ACT_RELU = 1, ACT_SIGMOID = 2, ACT_STEP = 3, ACT_TANH = 4 };

__device__ __forceinline__ float act_exp(float x) { return expf(x); }
__device__ __forceinline__ double act_exp(double x) { return exp(x); }
__device__ __forceinline__ float act_tanh(float x) { return tanhf(x); }
__device__ __forceinline__ double act_tanh(double x) { return tanh(x); }
__device__ __forceinline__ float act_abs(float x) { return fabsf(x); }
__device__ __forceinline__ double act_abs(double x) { return fabs(x); }

// 1 / x for x in [1, 2]: the hardware reciprocal (within 1 ulp) and one
// Newton step, in place of the IEEE division sequence
__device__ __forceinline__ float act_rcp12(float x) {
  const float r = __builtin_amdgcn_rcpf(x);
  return fmaf(r, fmaf(-x, r, 1.0f), r);
}
__device__ __forceinline__ double act_rcp12(double x) { return 1.0 / x; }

// tanh(z) for |z| < 1/2 from its Taylor series about 0, odd powers up to
// z^15 (coefficients 2^2n (2^2n - 1) B_2n / (2n)!; the first term left out
// is about 1e-8 of tanh(z) at |z| = 1/2)
__device__ __forceinline__ float act_tanh_small(float z) {
  const float z2 = z * z;
  float q = -929569.0f / 638512875.0f;
  q = fmaf(z2, q, 21844.0f / 6081075.0f);
  q = fmaf(z2, q, -1382.0f / 155925.0f);
  q = fmaf(z2, q, 62.0f / 2835.0f);
  q = fmaf(z2, q, -17.0f / 315.0f);
  q = fmaf(z2, q, 2.0f / 15.0f);
  q = fmaf(z2, q, -1.0f / 3.0f);
  return fmaf(z * z2, q, z);
}

// f(z) and f'(z) of the five activations (section 2; sigmoid from section 3.1).
// The sigmoid and tanh derivatives are formed from exp(-|z|) so that they keep
// their relative accuracy when the unit saturates.  In fp32 tanh itself is
// formed from the same exponential, (1 - e) / (1 + e) with e = exp(-2|z|),
// except for |z| < 1/2 where 1 - e cancels and the series is used: one
// exponential and one reciprocal per unit, within 4 ulp of tanh (checked
// against fp64 tanh over [-20, 20]).  fp64 uses the library tanh.
template <class T>
__device__ __forceinline__ void act_eval(int act, T z, T& f, T& fp) {
  const T zero = T(0), one = T(1);
  switch (act) {
    case ACT_SIGMOID: {
      const T e = act_exp(-act_abs(z));
      const T r = act_rcp12(one + e);
      f = z >= zero ? r : e * r;
      fp = e * r * r;  // sigma(z) sigma(-z)
      break;
    }
    case ACT_TANH: {
      const T az = act_abs(z);
      const T e = act_exp(T(-2) * az);
      const T r = act_rcp12(one + e);
      if constexpr (sizeof(T) == 4) {
        // both forms for every z and a select: a branch would run both
        // wherever a wavefront holds pre-activations on both sides of 1/2
        const T small = act_tanh_small(z);
        const T big = copysignf((one - e) * r, z);
        f = az < T(0.5) ? small : big;
      } else {
        f = act_tanh(z);
      }
      fp = T(4) * e * r * r;  // 1 - tanh^2 = 4 e^{-2|z|} / (1 + e^{-2|z|})^2
      break;
    }
    case ACT_RELU:
      f = z > zero ? z : zero;
      fp = z > zero ? one : zero;
      break;
    case ACT_GAUSSIAN: {
      const T g = act_exp(-z * z);
      f = g;
      fp = T(-2) * z * g;
      break;
    }
    default:  // ACT_STEP
      f = z > zero ? one : zero;
      fp = zero;
      break;
  }
}

}  // namespace nf
