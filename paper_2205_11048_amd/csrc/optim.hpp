// Optimiser updates of one float32 element.  Table 1 of the paper names
// Adagrad and Adam; the rules are the textbook ones.  The dense updates and
// Adam compute in float64 and round once per stored value; the Adagrad update
// of table rows computes in float32 (below).
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

}  // namespace gba
