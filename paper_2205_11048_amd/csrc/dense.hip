// Dense part of the push-step: the decayed weighted sum of the K dense
// gradients divided by N_a (Alg. 2), and the elementwise optimiser updates
// (Adagrad, Adam; Table 1 names them).
//
// The reduction streams K_eff * P floats from HBM: one thread owns four
// consecutive elements, issues 16-byte non-temporal loads from several
// gradients at a time, and accumulates in float64 in buffer order, so the
// only rounding is the final one to float (the result does not depend on the
// order in which the hardware schedules the loads).
#include "gba_device.hpp"
#include "gba_internal.hpp"
#include "optim.hpp"

namespace gba {

constexpr int kDenseBlock = 256;
constexpr int kDenseUnroll = 8;
constexpr int64_t kDenseMaxBlocks = 8192;

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Every block builds, in LDS, the ordered list of contributions whose weight
// is non-zero; excluded gradients are never touched (Eq. 1: they are not
// aggregated).  `aligned` tells whether every kept gradient allows 16-byte loads.
__device__ __forceinline__ int build_kept_list(const float* const* grads, const float* w, int K,
                                               uint16_t* kept, float* kw, uint32_t* tmp,
                                               int* aligned) {
  constexpr int kPer = (GBA_MAX_K + kDenseBlock - 1) / kDenseBlock;
  const int lo = threadIdx.x * kPer;
  uint32_t c = 0;
  bool al = true;
  for (int k = 0; k < kPer; ++k) {
    const int m = lo + k;
    if (m < K && w[m] != 0.0f) {
      ++c;
      al &= ((reinterpret_cast<uintptr_t>(grads[m]) & 15u) == 0);
    }
  }
  if (threadIdx.x == 0) *aligned = 1;
  __syncthreads();
  if (!al) *aligned = 0;
  uint32_t total;
  uint32_t pos = block_exclusive_scan<kDenseBlock>(c, tmp, &total);
  for (int k = 0; k < kPer; ++k) {
    const int m = lo + k;
    if (m < K && w[m] != 0.0f) {
      kept[pos] = (uint16_t)m;
      kw[pos] = w[m];
      ++pos;
    }
  }
  __syncthreads();
  return (int)total;
}

__global__ void __launch_bounds__(kDenseBlock)
aggregate_dense_kernel(const float* const* __restrict__ grads, const float* __restrict__ w, int K,
                       int64_t P, float* __restrict__ out) {
  __shared__ uint16_t kept[GBA_MAX_K];
  __shared__ float kw[GBA_MAX_K];
  __shared__ uint32_t tmp[kDenseBlock / kWave + 1];
  __shared__ int aligned;
  const int nk = build_kept_list(grads, w, K, kept, kw, tmp, &aligned);
  const double denom = (double)K;
  const int64_t stride = (int64_t)gridDim.x * kDenseBlock;
  if (aligned) {
    const int64_t nvec = P / 4;
    for (int64_t v = (int64_t)blockIdx.x * kDenseBlock + threadIdx.x; v < nvec; v += stride) {
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      int i = 0;
      for (; i + kDenseUnroll <= nk; i += kDenseUnroll) {
        f32x4 x[kDenseUnroll];
#pragma unroll
        for (int u = 0; u < kDenseUnroll; ++u)
          x[u] = load_stream(reinterpret_cast<const f32x4*>(grads[kept[i + u]]) + v);
#pragma unroll
        for (int u = 0; u < kDenseUnroll; ++u) acc += (double)kw[i + u] * widen(x[u]);
      }
      for (; i < nk; ++i)
        acc += (double)kw[i] * widen(load_stream(reinterpret_cast<const f32x4*>(grads[kept[i]]) + v));
      store_stream(reinterpret_cast<f32x4*>(out) + v, narrow(acc / denom));
    }
    // the last P % 4 elements
    const int64_t tail0 = nvec * 4;
    if (blockIdx.x == 0 && threadIdx.x < P - tail0) {
      const int64_t e = tail0 + threadIdx.x;
      double acc = 0.0;
      for (int i = 0; i < nk; ++i) acc += (double)kw[i] * (double)grads[kept[i]][e];
      out[e] = (float)(acc / denom);
    }
  } else {
    for (int64_t e = (int64_t)blockIdx.x * kDenseBlock + threadIdx.x; e < P; e += stride) {
      double acc = 0.0;
      for (int i = 0; i < nk; ++i) acc += (double)kw[i] * (double)grads[kept[i]][e];
      out[e] = (float)(acc / denom);
    }
  }
}

hipError_t launch_aggregate_dense(const float* const* grads, const float* w, int32_t K, int64_t P,
                                  float* out, hipStream_t stream) {
  if (P <= 0) return hipSuccess;
  int64_t blocks = ceil_div(ceil_div(P, 4), kDenseBlock);
  if (blocks > kDenseMaxBlocks) blocks = kDenseMaxBlocks;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(aggregate_dense_kernel, dim3((unsigned)blocks), dim3(kDenseBlock), 0, stream,
                     grads, w, (int)K, P, out);
  return hipGetLastError();
}

// ---------------------------------------------------------------- optimisers
__global__ void __launch_bounds__(kDenseBlock)
dense_adagrad_kernel(float* __restrict__ p, float* __restrict__ a, const float* __restrict__ g,
                     int64_t n, double lr, double eps) {
  const int64_t stride = (int64_t)gridDim.x * kDenseBlock;
  for (int64_t e = (int64_t)blockIdx.x * kDenseBlock + threadIdx.x; e < n; e += stride) {
    float pe = p[e], ae = a[e];
    adagrad_update(pe, ae, g[e], lr, eps);
    p[e] = pe;
    a[e] = ae;
  }
}

__global__ void __launch_bounds__(kDenseBlock)
dense_adam_kernel(float* __restrict__ p, float* __restrict__ m, float* __restrict__ v,
                  const float* __restrict__ g, int64_t n, double lr, double b1, double b2,
                  double eps, double bc1, double bc2) {
  const int64_t stride = (int64_t)gridDim.x * kDenseBlock;
  for (int64_t e = (int64_t)blockIdx.x * kDenseBlock + threadIdx.x; e < n; e += stride) {
    float pe = p[e], me = m[e], ve = v[e];
    adam_update(pe, me, ve, g[e], lr, b1, b2, eps, bc1, bc2);
    p[e] = pe;
    m[e] = me;
    v[e] = ve;
  }
}

hipError_t launch_dense_adagrad(float* p, float* a, const float* g, int64_t n, double lr, double eps,
                                hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = ceil_div(n, kDenseBlock);
  if (blocks > kDenseMaxBlocks) blocks = kDenseMaxBlocks;
  hipLaunchKernelGGL(dense_adagrad_kernel, dim3((unsigned)blocks), dim3(kDenseBlock), 0, stream, p,
                     a, g, n, lr, eps);
  return hipGetLastError();
}

hipError_t launch_dense_adam(float* p, float* m, float* v, const float* g, int64_t n,
                             const AdamParams& hp, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = ceil_div(n, kDenseBlock);
  if (blocks > kDenseMaxBlocks) blocks = kDenseMaxBlocks;
  hipLaunchKernelGGL(dense_adam_kernel, dim3((unsigned)blocks), dim3(kDenseBlock), 0, stream, p, m,
                     v, g, n, hp.lr, hp.beta1, hp.beta2, hp.eps, hp.bc1, hp.bc2);
  return hipGetLastError();
}

}  // namespace gba
