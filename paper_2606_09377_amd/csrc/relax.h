// ReLU linear relaxation (paper, Sec. 2.1, CROWN), shared by the device kernels that turn
// pre-activation bounds [l, u] into relaxation parameters.  Device code only.
//
// On [l, u] a ReLU is bounded by lam z <= ReLU(z) <= s z + t:
//   u <= 0 : inactive, (lam, s, t) = (0, 0, 0);   l >= 0 : active, (1, 1, 0);
//   else   : s = u / (u - l), t = -s l (the chord through (l, 0) and (u, u)) and a lower
//            slope lam in [0, 1].  Any lam in [0, 1] is sound; the rule that picks it:
//            adaptive (the default): 1 if u > -l else 0 (a tie gives 0); zero; one;
//            same slope: lam = s.
// The parameters are packed as float4 (lam, s, t, b) with b the bias that the backward
// pass adds next.
#pragma once

#include <hip/hip_runtime.h>

namespace vcr {

// values of VCR_OPT_LAMBDA_RULE
enum LambdaRule : int { LAMBDA_ADAPTIVE = 0, LAMBDA_ZERO = 1, LAMBDA_ONE = 2, LAMBDA_SAME_SLOPE = 3 };

__device__ __forceinline__ float4 relax_params(float l, float u, float bias, int rule) {
  if (u <= 0.f) return make_float4(0.f, 0.f, 0.f, bias);
  if (l >= 0.f) return make_float4(1.f, 1.f, 0.f, bias);
  const float s = u / (u - l);
  const float t = -s * l;
  float lam;
  switch (rule) {
    case LAMBDA_ZERO: lam = 0.f; break;
    case LAMBDA_ONE: lam = 1.f; break;
    case LAMBDA_SAME_SLOPE: lam = s; break;
    default: lam = (u > -l) ? 1.f : 0.f; break;
  }
  return make_float4(lam, s, t, bias);
}

}  // namespace vcr
