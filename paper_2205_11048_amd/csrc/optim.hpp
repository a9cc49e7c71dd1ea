// Optimiser updates of one float32 element, computed in float64 and rounded
// once per stored value.  Table 1 of the paper names Adagrad and Adam; the
// rules are the textbook ones.
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
