// Device twin of synth/counter.py: fills device arrays with the same
// counter-based values (SplitMix64 output number (stream << 40) + index of
// the generator seeded with `seed`; Steele, Lea and Flood, OOPSLA 2014), so
// arrays too large for the host can be made in place and any element
// re-derived on the host.  Holds no step of the aggregation method.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;

__device__ __forceinline__ uint64_t mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__device__ __forceinline__ uint64_t word(uint64_t seed, uint32_t stream, uint64_t index) {
  const uint64_t ctr = ((uint64_t)stream << 40) + index;
  return mix(seed + (ctr + 1ull) * kGamma);
}

// kinds: 0 param, 1 accum, 2 adam_m, 3 adam_v, 4 grad, 5 dyadic
__device__ __forceinline__ float value(uint64_t w, int kind, float scale) {
  const int64_t u24 = (int64_t)(w >> 40);
  switch (kind) {
    case 0: return (float)(u24 - (1 << 23)) * 0x1p-27f;
    case 1: return (float)(u24 + (1 << 22)) * 0x1p-26f;
    case 2: return (float)(u24 - (1 << 23)) * 0x1p-33f;
    case 3: return (float)(u24 + (1 << 22)) * 0x1p-40f;
    case 4: {
      const int64_t s = (int64_t)(w & 0xFFFF) + (int64_t)((w >> 16) & 0xFFFF) +
                        (int64_t)((w >> 32) & 0xFFFF) + (int64_t)(w >> 48) - 131070;
      return (float)s * scale;
    }
    default: return (float)((int64_t)(w >> 56) - 128) * 0x1p-8f;
  }
}

__global__ void fill_f32_kernel(float* __restrict__ out, int64_t n, uint64_t seed, uint32_t stream,
                                uint64_t start, int kind, float scale) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    out[i] = value(word(seed, stream, start + (uint64_t)i), kind, scale);
}

__global__ void fill_tags_kernel(int32_t* __restrict__ out, int64_t n, uint64_t seed, uint32_t stream,
                                 int64_t step) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const uint64_t w = word(seed, stream, (uint64_t)i);
    int64_t g = w == 0 ? 64 : __builtin_ctzll(w);
    g = g < 62 ? g : 62;
    int64_t t = step - 1 - g;
    t = t < -1 ? -1 : t;
    out[i] = (w >> 63) ? (int32_t)t : -1;
  }
}

inline unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 16384) b = 16384;
  return (unsigned)(b < 1 ? 1 : b);
}

}  // namespace

extern "C" int synth_fill_f32(float* out, int64_t n, uint64_t seed, uint32_t stream, uint64_t start,
                              int kind, float scale, hipStream_t s) {
  if (n <= 0) return 0;
  if (!out || kind < 0 || kind > 5 || stream >= (1u << 24)) return 1;
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(n)), dim3(256), 0, s, out, n, seed, stream, start,
                     kind, scale);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

extern "C" int synth_fill_tags(int32_t* out, int64_t n, uint64_t seed, uint32_t stream, int64_t step,
                               hipStream_t s) {
  if (n <= 0) return 0;
  if (!out || stream >= (1u << 24)) return 1;
  hipLaunchKernelGGL(fill_tags_kernel, dim3(grid_for(n)), dim3(256), 0, s, out, n, seed, stream, step);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}
