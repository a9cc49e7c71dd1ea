// Optimiser updates of one float32 element.  Table 1 of the paper names
// Adagrad and Adam; the rules are the textbook ones.  The dense updates
// compute in float64 and round once per stored value; the updates of
// embedding-table rows compute in float32 (the *_f32 forms below).
#pragma once

#include <hip/hip_runtime.h>

namespace gba {

// Adagrad (Duchi et al. 2011): a' = a + g^2; p' = p - lr g / (sqrt(a') + eps).
__device__ __forceinline__ void adagrad_update(float& p, float& a, float g, double lr, double eps) {
  const double gd = (double)g;
  const double an = (double)a + gd * gd;
  const double pn = (double)p - lr * gd / (sqrt(an) + eps);
  p = (float)pn;
  a = (float)an;
}

// Adagrad on embedding-table rows: the same rule in float32, with the
// hardware square root and reciprocal (v_sqrt_f32, v_rcp_f32: each within
// 1 ulp).  The step lr g / (sqrt(a') + eps) comes out within a few float32
// ulps of its exact value, and p' and a' take one rounding each, so the error
// is a few 1e-7 of |p| + |step| and of a'.  The row passes gather random rows
// and issue the update for every touched row: this form takes 8 instructions
// per element, the float64 one some 35, among them a correctly rounded
// float64 square root and division.
__device__ __forceinline__ void adagrad_update_f32(float& p, float& a, float g, float lr, float eps) {
  const float an = a + g * g;
  const float den = __builtin_amdgcn_sqrtf(an) + eps;
  p = p - (lr * g) * __builtin_amdgcn_rcpf(den);
  a = an;
}

// Adam (Kingma and Ba 2015) with bias corrections bc1 = 1 - b1^t, bc2 = 1 - b2^t.
__device__ __forceinline__ void adam_update(float& p, float& m, float& v, float g, double lr,
                                            double b1, double b2, double eps, double bc1,
                                            double bc2) {
  const double gd = (double)g;
  const double mn = b1 * (double)m + (1.0 - b1) * gd;
  const double vn = b2 * (double)v + (1.0 - b2) * gd * gd;
  const double mh = mn / bc1;
  const double vh = vn / bc2;
  const double pn = (double)p - lr * mh / (sqrt(vh) + eps);
  p = (float)pn;
  m = (float)mn;
  v = (float)vn;
}

// Adam on embedding-table rows in float32: the same rule with the hardware
// square root and reciprocal, the constants rounded once from double (omb1 =
// 1 - beta1, omb2 = 1 - beta2, rbc1 = 1 / bc1, rbc2 = 1 / bc2).  m' and v'
// are within a few float32 ulps of b1 |m| + (1 - b1) |g| and of v', the step
// within a few ulps of its value, and p' takes one more rounding.
__device__ __forceinline__ void adam_update_f32(float& p, float& m, float& v, float g, float lr, float b1,
                                                float omb1, float b2, float omb2, float eps, float rbc1,
                                                float rbc2) {
  const float mn = b1 * m + omb1 * g;
  const float vn = b2 * v + omb2 * (g * g);
  const float den = __builtin_amdgcn_sqrtf(vn * rbc2) + eps;
  p = p - (lr * (mn * rbc1)) * __builtin_amdgcn_rcpf(den);
  m = mn;
  v = vn;
}

}  // namespace gba
