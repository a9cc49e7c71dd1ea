// Device-wide exclusive prefix sum of uint32 counts (reduce, then scan).
// Used for the radix-sort digit offsets and for the segment numbering.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kScanBlock = 256;
constexpr int kScanItems = 8;
constexpr int64_t kScanTile = kScanBlock * kScanItems;

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

__global__ void __launch_bounds__(kScanBlock)
scan_reduce_kernel(const uint32_t* __restrict__ in, int64_t n, uint32_t* __restrict__ sums) {
  __shared__ uint32_t tmp[kScanBlock / kWave + 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  uint32_t s = 0;
  for (int k = 0; k < kScanItems; ++k) {
    const int64_t i = base + (int64_t)k * kScanBlock + threadIdx.x;
    if (i < n) s += in[i];
  }
  uint32_t total;
  block_exclusive_scan<kScanBlock>(s, tmp, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Scans one tile per block; thread t owns items [t * 8, t * 8 + 8) of the tile.
// `prefix` (may be null) holds the exclusive prefix of the tile totals.  The
// last block writes the grand total to *total when total is not null.
__global__ void __launch_bounds__(kScanBlock)
scan_tile_kernel(const uint32_t* in, uint32_t* out, int64_t n, const uint32_t* __restrict__ prefix,
                 uint32_t* __restrict__ total) {
  __shared__ uint32_t tmp[kScanBlock / kWave + 1];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  uint32_t v[kScanItems];
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int64_t i = base + k;
    v[k] = (i < n) ? in[i] : 0u;
    s += v[k];
  }
  uint32_t tile_total;
  uint32_t run = block_exclusive_scan<kScanBlock>(s, tmp, &tile_total);
  const uint32_t off = prefix ? prefix[blockIdx.x] : 0u;
  run += off;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const int64_t i = base + k;
    if (i < n) out[i] = run;
    run += v[k];
  }
  if (total && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *total = off + tile_total;
}

size_t scan_workspace_bytes(int64_t n) {
  size_t words = 0;
  int64_t m = n;
  while (m > kScanTile) {
    m = ceil_div(m, kScanTile);
    words += (size_t)m;
  }
  return words * sizeof(uint32_t) + 256;
}

hipError_t launch_exclusive_scan_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total,
                                     void* ws, hipStream_t stream) {
  if (n <= 0) {
    if (total) {
      hipLaunchKernelGGL(scan_tile_kernel, dim3(1), dim3(kScanBlock), 0, stream, in, out,
                         (int64_t)0, nullptr, total);
      return hipGetLastError();
    }
    return hipSuccess;
  }
  if (n <= kScanTile) {
    hipLaunchKernelGGL(scan_tile_kernel, dim3(1), dim3(kScanBlock), 0, stream, in, out, n, nullptr,
                       total);
    return hipGetLastError();
  }
  const int64_t nb = ceil_div(n, kScanTile);
  uint32_t* sums = static_cast<uint32_t*>(ws);
  hipLaunchKernelGGL(scan_reduce_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, in, n, sums);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_exclusive_scan_u32(sums, sums, nb, nullptr, sums + nb, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(scan_tile_kernel, dim3((unsigned)nb), dim3(kScanBlock), 0, stream, in, out, n,
                     sums, total);
  return hipGetLastError();
}

}  // namespace gba
