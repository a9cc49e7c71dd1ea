// Token weights of the K buffered contributions: Eq. 1 (Sec. 3.1).
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

// One block of up to 1024 threads walks the K tokens (K <= 4096).
__global__ void __launch_bounds__(1024)
token_weights_kernel(const int64_t* __restrict__ tokens, int32_t K, int64_t step, int64_t iota,
                     float* __restrict__ w, int64_t* __restrict__ staleness,
                     int32_t* __restrict__ num_excluded, int32_t* __restrict__ err) {
  __shared__ uint32_t tmp[1024 / kWave + 1];
  uint32_t excluded = 0;
  bool future = false;
  for (int m = threadIdx.x; m < K; m += blockDim.x) {
    const int64_t s = step - tokens[m];
    // f = 1 when the data staleness s is within the tolerance iota, else 0.
    const bool keep = (s >= 0) && (s <= iota);
    future |= (s < 0);
    w[m] = keep ? 1.0f : 0.0f;
    if (staleness) staleness[m] = s;
    excluded += keep ? 0u : 1u;
  }
  if (future) raise_error(err, GBA_DERR_FUTURE_TOKEN);
  uint32_t total;
  block_exclusive_scan<1024>(excluded, tmp, &total);
  if (threadIdx.x == 0 && num_excluded) *num_excluded = (int32_t)total;
}

hipError_t launch_token_weights(const int64_t* tokens, int32_t K, int64_t step, int64_t iota,
                                float* w, int64_t* staleness, int32_t* num_excluded, int32_t* err,
                                hipStream_t stream) {
  hipLaunchKernelGGL(token_weights_kernel, dim3(1), dim3(1024), 0, stream, tokens, K, step, iota,
                     w, staleness, num_excluded, err);
  return hipGetLastError();
}

}  // namespace gba
