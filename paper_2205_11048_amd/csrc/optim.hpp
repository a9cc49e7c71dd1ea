// Optimiser updates of one float32 element.  Table 1 of the paper names
// Adagrad and Adam; the rules are the textbook ones, computed in float32 from
// the float32 state and gradient, with the hardware square root and
// reciprocal (v_sqrt_f32, v_rcp_f32: each within 1 ulp) and the constants
// rounded once from double.  Each step then comes out within a few float32
// ulps of its exact value and every stored value takes one more rounding, so
// the error stays a few 1e-7 of the magnitude the values are built from
// (|p| + |step|, b1 |m| + (1 - b1) |g|, v').  The float64 forms (a correctly
// rounded float64 square root and division per element) cost the row passes
// a quarter of their instructions, and the dense reduction its finishing.
#pragma once

#include <hip/hip_runtime.h>

namespace gba {

// The float32 constants of one update: lr, eps, b1, 1 - b1, b2, 1 - b2,
// 1 / bc1, 1 / bc2 (bc1 = 1 - b1^t, bc2 = 1 - b2^t), each rounded once from
// double.  Adagrad reads lr and eps only.
struct OptF32 {
  float lr, eps, b1, omb1, b2, omb2, rbc1, rbc2;
};

__host__ __device__ inline OptF32 opt_f32(double lr, double eps, double b1 = 0.0, double b2 = 0.0,
                                          double bc1 = 1.0, double bc2 = 1.0) {
  return OptF32{(float)lr, (float)eps, (float)b1, (float)(1.0 - b1), (float)b2, (float)(1.0 - b2),
                (float)(1.0 / bc1), (float)(1.0 / bc2)};
}

// Adagrad (Duchi et al. 2011): a' = a + g^2; p' = p - lr g / (sqrt(a') + eps).
__device__ __forceinline__ void adagrad_update_f32(float& p, float& a, float g, const OptF32& c) {
  const float an = a + g * g;
  const float den = __builtin_amdgcn_sqrtf(an) + c.eps;
  p = p - (c.lr * g) * __builtin_amdgcn_rcpf(den);
  a = an;
}

// Adam (Kingma and Ba 2015): m' = b1 m + (1 - b1) g; v' = b2 v + (1 - b2) g^2;
// p' = p - lr (m' / bc1) / (sqrt(v' / bc2) + eps).
__device__ __forceinline__ void adam_update_f32(float& p, float& m, float& v, float g, const OptF32& c) {
  const float mn = c.b1 * m + c.omb1 * g;
  const float vn = c.b2 * v + c.omb2 * (g * g);
  const float den = __builtin_amdgcn_sqrtf(vn * c.rbc2) + c.eps;
  p = p - (c.lr * (mn * c.rbc1)) * __builtin_amdgcn_rcpf(den);
  m = mn;
  v = vn;
}

}  // namespace gba
