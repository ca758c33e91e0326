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

// f(z) and f'(z) of the five activations (section 2; sigmoid from section 3.1).
// The sigmoid and tanh derivatives are formed from exp(-|z|) so that they keep
// their relative accuracy when the unit saturates.
template <class T>
__device__ __forceinline__ void act_eval(int act, T z, T& f, T& fp) {
  const T zero = T(0), one = T(1);
  switch (act) {
    case ACT_SIGMOID: {
      const T e = act_exp(-act_abs(z));
      const T r = one / (one + e);
      f = z >= zero ? r : e * r;
      fp = e * r * r;  // sigma(z) sigma(-z)
      break;
    }
    case ACT_TANH: {
      f = act_tanh(z);
      const T e = act_exp(T(-2) * act_abs(z));
      const T r = one / (one + e);
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
