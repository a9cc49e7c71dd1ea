// Measurement kernels (declared in include/gba_ceilings.h): the bandwidth
// this GPU delivers for the access patterns of the push-step, each measured
// with the plainest kernel that has it.  Not part of the step.
#include "gba_ceilings.h"
#include "gba_device.hpp"

namespace gba {

constexpr int kCeilBlock = 256;
constexpr int kCeilUnroll = 8;   // vectors (or rows) in flight per lane
// the read stream: 4 vectors per lane (of the shapes tried, 256 or 512
// threads with 4, 8 or 16 vectors per lane, lane-consecutive or in runs of
// 1-16 KB per wave, at 512-16384 blocks, this one read fastest)
constexpr int kCeilReadUnroll = 4;
constexpr int kCeilWaves = kCeilBlock / kWave;

__device__ __forceinline__ uint32_t bits_of(f32x4 v) {
  return __float_as_uint(v.x) ^ __float_as_uint(v.y) ^ __float_as_uint(v.z) ^ __float_as_uint(v.w);
}

__device__ __forceinline__ void put_wave_word(uint32_t x, uint32_t* sink) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) x ^= __shfl_xor(x, off, kWave);
  if (lane_id() == 0) sink[(int64_t)blockIdx.x * kCeilWaves + threadIdx.x / kWave] = x;
}

// Each round a block reads kCeilReadUnroll * kCeilBlock consecutive vectors
// (16 KB), lane-consecutive, all loads issued before the first is used.
__global__ void __launch_bounds__(kCeilBlock)
ceiling_read_kernel(const f32x4* __restrict__ src, int64_t n, uint32_t* __restrict__ sink) {
  constexpr int64_t kSpan = (int64_t)kCeilBlock * kCeilReadUnroll;
  uint32_t x = 0;
  for (int64_t b = (int64_t)blockIdx.x * kSpan; b < n; b += (int64_t)gridDim.x * kSpan) {
    f32x4 v[kCeilReadUnroll];
#pragma unroll
    for (int u = 0; u < kCeilReadUnroll; ++u) {
      const int64_t i = b + (int64_t)u * kCeilBlock + threadIdx.x;
      v[u] = i < n ? load_stream(src + i) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < kCeilReadUnroll; ++u) x ^= bits_of(v[u]);
  }
  put_wave_word(x, sink);
}

__global__ void __launch_bounds__(kCeilBlock)
ceiling_copy_kernel(const f32x4* __restrict__ src, f32x4* __restrict__ dst, int64_t n) {
  constexpr int64_t kSpan = (int64_t)kCeilBlock * kCeilUnroll;
  for (int64_t b = (int64_t)blockIdx.x * kSpan; b < n; b += (int64_t)gridDim.x * kSpan) {
    f32x4 v[kCeilUnroll];
#pragma unroll
    for (int u = 0; u < kCeilUnroll; ++u) {
      const int64_t i = b + (int64_t)u * kCeilBlock + threadIdx.x;
      if (i < n) v[u] = load_stream(src + i);
    }
#pragma unroll
    for (int u = 0; u < kCeilUnroll; ++u) {
      const int64_t i = b + (int64_t)u * kCeilBlock + threadIdx.x;
      if (i < n) store_stream(dst + i, v[u]);
    }
  }
}

// Lane group g of G = D/4 lanes (64 / G groups per wave; lanes past the last
// whole group idle) takes one row per slot, kCeilUnroll slots per round.
__global__ void __launch_bounds__(kCeilBlock)
ceiling_gather_kernel(const float* __restrict__ table, int64_t R, int D, const int64_t* __restrict__ rows, int64_t n,
                      uint32_t* __restrict__ sink) {
  const int G = D / 4;
  const int groups = kWave / G;
  const int lane = lane_id();
  const int g = lane / G, c = lane % G;
  const bool on = g < groups;
  const int64_t wave = ((int64_t)blockIdx.x * kCeilBlock + threadIdx.x) / kWave;
  const int64_t waves = (int64_t)gridDim.x * kCeilWaves;
  const int64_t per_round = (int64_t)groups * kCeilUnroll;
  uint32_t x = 0;
  for (int64_t b = wave * per_round; b < n; b += waves * per_round) {
    int64_t r[kCeilUnroll];
#pragma unroll
    for (int u = 0; u < kCeilUnroll; ++u) {
      const int64_t i = b + (int64_t)u * groups + g;
      r[u] = (on && i < n) ? rows[i] : -1;
    }
    f32x4 v[kCeilUnroll];
#pragma unroll
    for (int u = 0; u < kCeilUnroll; ++u) {
      const bool ok = r[u] >= 0 && r[u] < R;
      v[u] = ok ? *reinterpret_cast<const f32x4*>(table + r[u] * D + 4 * c) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int u = 0; u < kCeilUnroll; ++u) x ^= bits_of(v[u]);
  }
  put_wave_word(x, sink);
}

}  // namespace gba

using namespace gba;

namespace {
bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
gba_status launched() { return hipGetLastError() == hipSuccess ? GBA_OK : GBA_ERR_HIP; }
}  // namespace

extern "C" {

int64_t gba_ceiling_sink_words(int32_t blocks) { return blocks > 0 ? (int64_t)blocks * kCeilWaves : 0; }

gba_status gba_ceiling_read(const void* src, int64_t n16, uint32_t* sink, int32_t blocks, hipStream_t stream) {
  if (n16 < 0 || blocks < 1) return GBA_ERR_INVALID_ARG;
  if (!sink || (n16 > 0 && !src)) return GBA_ERR_NULL;
  if (src && !aligned16(src)) return GBA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(ceiling_read_kernel, dim3((unsigned)blocks), dim3(kCeilBlock), 0, stream,
                     static_cast<const f32x4*>(src), n16, sink);
  return launched();
}

gba_status gba_ceiling_copy(const void* src, void* dst, int64_t n16, int32_t blocks, hipStream_t stream) {
  if (n16 < 0 || blocks < 1) return GBA_ERR_INVALID_ARG;
  if (n16 == 0) return GBA_OK;
  if (!src || !dst) return GBA_ERR_NULL;
  if (!aligned16(src) || !aligned16(dst)) return GBA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(ceiling_copy_kernel, dim3((unsigned)blocks), dim3(kCeilBlock), 0, stream,
                     static_cast<const f32x4*>(src), static_cast<f32x4*>(dst), n16);
  return launched();
}

gba_status gba_ceiling_gather_rows(const float* table, int64_t R, int32_t D, const int64_t* rows, int64_t n,
                                   uint32_t* sink, int32_t blocks, hipStream_t stream) {
  if (n < 0 || blocks < 1 || R < 1) return GBA_ERR_INVALID_ARG;
  if (D < 4 || D > GBA_MAX_D || D % 4 != 0) return GBA_ERR_UNSUPPORTED;
  if (!sink || (n > 0 && (!table || !rows))) return GBA_ERR_NULL;
  if (table && !aligned16(table)) return GBA_ERR_INVALID_ARG;
  hipLaunchKernelGGL(ceiling_gather_kernel, dim3((unsigned)blocks), dim3(kCeilBlock), 0, stream, table, R, (int)D,
                     rows, n, sink);
  return launched();
}

}  // extern "C"
