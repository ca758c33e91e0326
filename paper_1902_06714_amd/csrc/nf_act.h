// f(z) and f'(z) of the activation functions, shared by the device kernels.
#pragma once

#include <hip/hip_runtime.h>

namespace nf {

enum { ACT_GAUSSIAN = 0, ACT_RELU = 1, ACT_SIGMOID = 2, ACT_STEP = 3, ACT_TANH = 4 };

// f(z) and f'(z) of the five activations (section 2; sigmoid from section 3.1).
// The sigmoid and tanh derivatives are formed from exp(-|z|) so that they keep
// their relative accuracy when the unit saturates.
__device__ __forceinline__ void act_eval(int act, float z, float& f, float& fp) {
  switch (act) {
    case ACT_SIGMOID: {
      const float e = expf(-fabsf(z));
      const float r = 1.0f / (1.0f + e);
      f = z >= 0.0f ? r : e * r;
      fp = e * r * r;  // sigma(z) sigma(-z)
      break;
    }
    case ACT_TANH: {
      f = tanhf(z);
      const float e = expf(-2.0f * fabsf(z));
      const float r = 1.0f / (1.0f + e);
      fp = 4.0f * e * r * r;  // 1 - tanh^2 = 4 e^{-2|z|} / (1 + e^{-2|z|})^2
      break;
    }
    case ACT_RELU:
      f = z > 0.0f ? z : 0.0f;
      fp = z > 0.0f ? 1.0f : 0.0f;
      break;
    case ACT_GAUSSIAN: {
      const float g = expf(-z * z);
      f = g;
      fp = -2.0f * z * g;
      break;
    }
    default:  // ACT_STEP
      f = z > 0.0f ? 1.0f : 0.0f;
      fp = 0.0f;
      break;
  }
}

}  // namespace nf
