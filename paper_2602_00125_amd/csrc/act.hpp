// Nonlinearities of MiniTensor Sec. 3.3 and their derivatives, in fp32 on
// the device: used by the GEMM epilogue (forward, applied to the biased
// product while it is still in registers) and by the elementwise pullback
// kernel (derivative at the saved pre-activation).
//
//   ReLU     max(z, 0)                 derivative: the indicator of z > 0
//   Sigmoid  1 / (1 + e^-z)            s (1 - s)
//   Tanh     tanh z                    1 - tanh^2 z
//   GELU     z Phi(z),                 Phi(z) + z phi(z)
//            Phi(z) = (1 + erf(z / sqrt 2)) / 2, phi(z) = e^(-z^2/2) / sqrt(2 pi)
//
// erff, expf and tanhf are the device library's fp32 functions (a few ulp).
#pragma once
#include <hip/hip_runtime.h>

namespace mt {

enum ActKind { kActNone = 0, kActRelu = 1, kActSigmoid = 2, kActTanh = 3, kActGelu = 4 };
constexpr int kNumAct = 5;

template <int ACT>
__device__ __forceinline__ float act_apply_t(float z) {
  if constexpr (ACT == kActRelu) return z > 0.f ? z : 0.f;
  else if constexpr (ACT == kActSigmoid) return 1.f / (1.f + expf(-z));
  else if constexpr (ACT == kActTanh) return tanhf(z);
  else if constexpr (ACT == kActGelu) return 0.5f * z * (1.f + erff(z * 0.70710678118654752f));
  else return z;
}

__device__ __forceinline__ float act_grad(int act, float z) {
  switch (act) {
    case kActRelu: return z > 0.f ? 1.f : 0.f;
    case kActSigmoid: {
      const float s = 1.f / (1.f + expf(-z));
      return s * (1.f - s);
    }
    case kActTanh: {
      const float t = tanhf(z);
      return 1.f - t * t;
    }
    case kActGelu: {
      const float cdf = 0.5f * (1.f + erff(z * 0.70710678118654752f));
      const float pdf = expf(-0.5f * z * z) * 0.39894228040143268f;
      return cdf + z * pdf;
    }
    default: return 1.f;
  }
}

}  // namespace mt
