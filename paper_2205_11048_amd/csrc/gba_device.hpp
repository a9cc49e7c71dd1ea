// Device-side building blocks shared by the GBA kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gba {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Inclusive scan of one 32-bit value across the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  const int l = lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    uint32_t y = __shfl_up(x, off, kWave);
    if (l >= off) x += y;
  }
  return x;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  return x;
}

// Exclusive scan over a block of BLOCK threads (BLOCK a multiple of 64, <= 1024).
// `tmp` must hold BLOCK / 64 + 1 words of LDS.  Returns the exclusive prefix;
// the block total is written to *total (every thread sees it).
template <int BLOCK>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* tmp, uint32_t* total) {
  constexpr int NW = BLOCK / kWave;
  const int w = threadIdx.x / kWave;
  const uint32_t inc = wave_inclusive_scan(x);
  if (lane_id() == kWave - 1) tmp[w] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int i = 0; i < NW; ++i) {
      uint32_t t = tmp[i];
      tmp[i] = run;
      run += t;
    }
    tmp[NW] = run;
  }
  __syncthreads();
  const uint32_t ex = tmp[w] + inc - x;
  *total = tmp[NW];
  __syncthreads();
  return ex;
}

// OR bits into the caller's device error word (vector atomic; rare path).
__device__ __forceinline__ void raise_error(int32_t* err, int32_t bits) {
  if (err) atomicOr(err, bits);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Loads and stores marked non-temporal, for data touched exactly once.
__device__ __forceinline__ f32x4 load_stream(const f32x4* p) { return __builtin_nontemporal_load(p); }
// The same from a pointer known to be in device global memory: a global (not
// flat) load, counted by the vector-memory counter only, so that waiting for
// an LDS or scalar load does not also wait for it.
typedef __attribute__((address_space(1))) const f32x4 global_f32x4;
__device__ __forceinline__ f32x4 load_stream_global(const f32x4* p) {
  return __builtin_nontemporal_load((global_f32x4*)p);
}
__device__ __forceinline__ void store_stream(f32x4* p, f32x4 v) { __builtin_nontemporal_store(v, p); }

__device__ __forceinline__ f64x4 widen(f32x4 v) {
  return f64x4{(double)v.x, (double)v.y, (double)v.z, (double)v.w};
}
// acc + w * x for a float32 weight w (widened) and a float32 row x: the
// product of two float32 values is exact in float64, so one fused
// multiply-add rounds exactly as the product followed by the sum does.
__device__ __forceinline__ f64x4 fma_widen(double w, f32x4 x, f64x4 acc) {
  return f64x4{__builtin_fma(w, (double)x.x, acc.x), __builtin_fma(w, (double)x.y, acc.y),
               __builtin_fma(w, (double)x.z, acc.z), __builtin_fma(w, (double)x.w, acc.w)};
}
__device__ __forceinline__ f32x4 narrow(f64x4 v) {
  return f32x4{(float)v.x, (float)v.y, (float)v.z, (float)v.w};
}

// acc / d for each element, rounded once, as a float64 division rounds it,
// at one division per vector instead of four: with y the rounded reciprocal
// of d and q = acc * y rounded (within an ulp of the quotient), the residual
// acc - q * d is exact in one fma and q + residual * y, rounded, is the
// rounded quotient (Markstein's theorem; Muller et al., Handbook of
// Floating-Point Arithmetic, the chapter on division by iteration).  It holds
// away from the float64 underflow and overflow ranges, far from sums of
// float32 values divided by a count.  y must be the rounded 1 / d.
__device__ __forceinline__ f64x4 div_rounded(f64x4 acc, double d, double y) {
  f64x4 q;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const double q0 = acc[e] * y;
    const double r = __builtin_fma(-q0, d, acc[e]);
    q[e] = __builtin_fma(r, y, q0);
  }
  return q;
}
__device__ __forceinline__ f64x4 div_rounded(f64x4 acc, double d) { return div_rounded(acc, d, 1.0 / d); }

}  // namespace gba
