// Stable LSD radix sort of the occurrence IDs, keyed by ID, carrying the
// occurrence index.  It groups the occurrences of each embedding ID so the
// push-step can deduplicate them and reduce their rows (Alg. 2: gradients of
// the embedding parameters are processed by ID).
//
// Each 8-bit digit takes three steps: a histogram per tile of 4096 keys
// (written tile-major, 1 KB per tile), a column scan that turns the per-tile
// counts into each tile's global offset per digit value (tile-major again, so
// a tile reads its 256 offsets as one contiguous line), and a scatter that
// ranks the tile stably in LDS and writes runs of equal digits together.
// Ranks inside a wave come from ballots that match lanes holding the same
// digit, so skewed (Zipf) keys cost no LDS atomics on hot bins in the scatter.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kSortBlock = 256;
constexpr int kSortWaves = kSortBlock / kWave;
constexpr int kSortItems = 16;                         // per lane
constexpr int kSortWaveTile = kWave * kSortItems;      // 1024 keys per wave
constexpr int64_t kSortTile = kSortBlock * kSortItems; // 4096 keys per tile
constexpr int kRadix = 256;
constexpr int kChunk = 32;                             // tiles per column-scan chunk

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

struct SortLayout {
  size_t arr, off_keys0, off_keys1, off_vals0, off_vals1, off_hist, off_chunk, off_base, bytes;
};

static SortLayout sort_layout(int64_t n, int64_t tiles) {
  SortLayout L{};
  L.arr = align_up((size_t)(n > 0 ? n : 1) * sizeof(uint32_t));
  const size_t nt = (size_t)(tiles > 0 ? tiles : 1);
  size_t o = 0;
  L.off_keys0 = o; o += L.arr;
  L.off_keys1 = o; o += L.arr;
  L.off_vals0 = o; o += L.arr;
  L.off_vals1 = o; o += L.arr;
  L.off_hist = o;  o += align_up(nt * kRadix * 4);                       // [tile][digit]
  L.off_chunk = o; o += align_up((size_t)ceil_div((int64_t)nt, kChunk) * kRadix * 4);
  L.off_base = o;  o += align_up(kRadix * 4);
  L.bytes = o;
  return L;
}

// Mask of the active lanes whose digit equals this lane's digit.
__device__ __forceinline__ uint64_t match_digit(uint32_t digit, int bits, bool active) {
  uint64_t m = __ballot(active);
  for (int b = 0; b < bits; ++b) {
    const bool bit = (digit >> b) & 1u;
    const uint64_t bal = __ballot(bit);
    m &= bit ? bal : ~bal;
  }
  return active ? m : 0ull;
}

// Key of position i: from the int64 IDs on the first pass (checked against
// [0, R); an ID outside it is reported and sorted as 0), else the u32 keys.
template <bool FIRST>
__device__ __forceinline__ uint32_t load_key(const void* src, int64_t i, int64_t R, bool* bad) {
  if (FIRST) {
    const int64_t id = static_cast<const int64_t*>(src)[i];
    if (id < 0 || id >= R) {
      *bad = true;
      return 0u;
    }
    return (uint32_t)id;
  }
  return static_cast<const uint32_t*>(src)[i];
}

// Digit counts of one tile, one 1 KB row per tile.  Each wave adds one count
// per run of equal digits among its 64 lanes, so the long runs of a hot ID
// (contiguous after the first pass) cost one LDS add, not 64 colliding ones.
template <bool FIRST>
__global__ void __launch_bounds__(kSortBlock)
sort_tile_hist_kernel(const void* __restrict__ keys_in, int64_t n, int shift, int bits, int64_t R,
                      uint32_t* __restrict__ hist, int32_t* __restrict__ err) {
  __shared__ uint32_t h[kSortWaves][kRadix];
  for (int i = threadIdx.x; i < kSortWaves * kRadix; i += kSortBlock) (&h[0][0])[i] = 0u;
  __syncthreads();
  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  const int64_t base = (int64_t)blockIdx.x * kSortTile + (int64_t)w * kSortWaveTile + lane;
  const uint32_t mask = (1u << bits) - 1u;
  bool bad = false;
  uint32_t digit[kSortItems];
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t i = base + (int64_t)r * kWave;
    digit[r] = i < n ? (load_key<FIRST>(keys_in, i, R, &bad) >> shift) & mask : 0u;
  }
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const bool active = base + (int64_t)r * kWave < n;   // active lanes are a prefix of the wave
    const uint32_t prev = __shfl_up(digit[r], 1, kWave);
    const bool head = active && (lane == 0 || digit[r] != prev);
    const uint64_t heads = __ballot(head);
    const int na = __popcll(__ballot(active));
    if (head) {
      const uint64_t above = lane == 63 ? 0ull : heads & (~0ull << (lane + 1));
      const int next = above ? __builtin_ctzll(above) : na;
      atomicAdd(&h[w][digit[r]], (uint32_t)(next - lane));
    }
  }
  if (FIRST && bad) raise_error(err, GBA_DERR_ID_RANGE);
  __syncthreads();
  const int d = threadIdx.x;   // kSortBlock == kRadix
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kSortWaves; ++k) s += h[k][d];
  hist[(int64_t)blockIdx.x * kRadix + d] = s;
}

// Column sums of chunks of kChunk tiles (the rows are read together).
__global__ void __launch_bounds__(kSortBlock)
sort_chunk_sum_kernel(const uint32_t* __restrict__ hist, int64_t tiles, uint32_t* __restrict__ chunk) {
  const int d = threadIdx.x;
  const int64_t t0 = (int64_t)blockIdx.x * kChunk;
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kChunk; ++k)
    if (t0 + k < tiles) s += hist[(t0 + k) * kRadix + d];
  chunk[(int64_t)blockIdx.x * kRadix + d] = s;
}

// Per digit: exclusive prefix over chunks; across digits: where each digit starts.
__global__ void __launch_bounds__(kSortBlock)
sort_chunk_scan_kernel(uint32_t* __restrict__ chunk, int64_t nchunks, uint32_t* __restrict__ base) {
  constexpr int kStep = 16;
  __shared__ uint32_t tmp[kSortBlock / kWave + 1];
  const int d = threadIdx.x;
  uint32_t run = 0;
  for (int64_t c0 = 0; c0 < nchunks; c0 += kStep) {
    uint32_t v[kStep];
#pragma unroll
    for (int k = 0; k < kStep; ++k) v[k] = (c0 + k < nchunks) ? chunk[(c0 + k) * kRadix + d] : 0u;
#pragma unroll
    for (int k = 0; k < kStep; ++k) {
      if (c0 + k < nchunks) chunk[(c0 + k) * kRadix + d] = run;
      run += v[k];
    }
  }
  uint32_t total;
  base[d] = block_exclusive_scan<kSortBlock>(run, tmp, &total);
}

// hist[tile][d] becomes the global position of the tile's first key with digit d.
__global__ void __launch_bounds__(kSortBlock)
sort_chunk_apply_kernel(uint32_t* __restrict__ hist, int64_t tiles, const uint32_t* __restrict__ chunk,
                        const uint32_t* __restrict__ base) {
  const int d = threadIdx.x;
  const int64_t t0 = (int64_t)blockIdx.x * kChunk;
  uint32_t run = base[d] + chunk[(int64_t)blockIdx.x * kRadix + d];
  uint32_t v[kChunk];
#pragma unroll
  for (int k = 0; k < kChunk; ++k) v[k] = (t0 + k < tiles) ? hist[(t0 + k) * kRadix + d] : 0u;
#pragma unroll
  for (int k = 0; k < kChunk; ++k) {
    if (t0 + k < tiles) hist[(t0 + k) * kRadix + d] = run;
    run += v[k];
  }
}

template <bool FIRST>
__global__ void __launch_bounds__(kSortBlock)
sort_scatter_kernel(const void* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
                    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t n,
                    int shift, int bits, int64_t R, const uint32_t* __restrict__ offsets) {
  __shared__ uint32_t cnt[kSortWaves][kRadix];
  __shared__ uint32_t digit_start[kRadix];
  __shared__ uint32_t global_base[kRadix];
  __shared__ uint32_t tmp[kSortBlock / kWave + 1];
  __shared__ uint32_t s_keys[kSortTile];
  __shared__ uint32_t s_vals[kSortTile];
  for (int i = threadIdx.x; i < kSortWaves * kRadix; i += kSortBlock) (&cnt[0][0])[i] = 0;
  global_base[threadIdx.x] = offsets[(int64_t)blockIdx.x * kRadix + threadIdx.x];
  __syncthreads();
  const int w = threadIdx.x / kWave;
  const int64_t tile0 = (int64_t)blockIdx.x * kSortTile;
  const int64_t base = tile0 + (int64_t)w * kSortWaveTile + lane_id();
  const uint32_t mask = (1u << bits) - 1u;
  const uint64_t lt = lanemask_lt();

  uint32_t key[kSortItems], val[kSortItems], rank[kSortItems];
  bool bad = false;
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t i = base + (int64_t)r * kWave;
    const bool active = i < n;
    key[r] = active ? load_key<FIRST>(keys_in, i, R, &bad) : 0u;
    val[r] = active ? (FIRST ? (uint32_t)i : vals_in[i]) : 0u;
  }
  (void)bad;   // range errors are reported by the histogram launch
  // Stable rank within (wave, digit): rounds in index order, lanes in order.
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t i = base + (int64_t)r * kWave;
    const bool active = i < n;
    const uint32_t digit = (key[r] >> shift) & mask;
    const uint64_t m = match_digit(digit, bits, active);
    uint32_t before = 0;
    if (active) before = cnt[w][digit];
    // every lane of the wave has read the counter before the leader updates it
    __builtin_amdgcn_wave_barrier();
    if (active && (m & lt) == 0) cnt[w][digit] = before + (uint32_t)__popcll(m);
    rank[r] = before + (uint32_t)__popcll(m & lt);
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();
  {
    const int d = threadIdx.x;
    uint32_t c[kSortWaves];
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      c[k] = cnt[k][d];
      s += c[k];
    }
    uint32_t total;
    const uint32_t ex = block_exclusive_scan<kSortBlock>(s, tmp, &total);
    digit_start[d] = ex;
    uint32_t run = ex;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      cnt[k][d] = run;
      run += c[k];
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t i = base + (int64_t)r * kWave;
    if (i < n) {
      const uint32_t digit = (key[r] >> shift) & mask;
      const uint32_t pos = cnt[w][digit] + rank[r];
      s_keys[pos] = key[r];
      s_vals[pos] = val[r];
    }
  }
  __syncthreads();
  const int64_t tile_n = (n - tile0) < kSortTile ? (n - tile0) : kSortTile;
  for (int i = threadIdx.x; i < tile_n; i += kSortBlock) {
    const uint32_t k = s_keys[i];
    const uint32_t digit = (k >> shift) & mask;
    const uint32_t g = global_base[digit] + ((uint32_t)i - digit_start[digit]);
    if ((int64_t)g < n) {   // always true when the counts are consistent
      keys_out[g] = k;
      vals_out[g] = s_vals[i];
    }
  }
}

SortPlan plan_sort(int64_t n, int64_t R) {
  SortPlan p{};
  p.n = n;
  int bits = 1;
  while (bits < 32 && ((int64_t)1 << bits) < R) ++bits;
  p.key_bits = bits;
  p.passes = (bits + 7) / 8;
  p.blocks = n > 0 ? ceil_div(n, kSortTile) : 0;
  p.bytes = sort_layout(n, p.blocks).bytes;
  return p;
}

hipError_t launch_sort_ids(const int64_t* ids, int64_t n, int64_t R, const SortPlan& plan, void* ws,
                           const uint32_t** keys_out, const uint32_t** vals_out, int32_t* err,
                           hipStream_t stream) {
  const SortLayout L = sort_layout(n, plan.blocks);
  char* p = static_cast<char*>(ws);
  uint32_t* keys[2] = {reinterpret_cast<uint32_t*>(p + L.off_keys0), reinterpret_cast<uint32_t*>(p + L.off_keys1)};
  uint32_t* vals[2] = {reinterpret_cast<uint32_t*>(p + L.off_vals0), reinterpret_cast<uint32_t*>(p + L.off_vals1)};
  uint32_t* hist = reinterpret_cast<uint32_t*>(p + L.off_hist);
  uint32_t* chunk = reinterpret_cast<uint32_t*>(p + L.off_chunk);
  uint32_t* base = reinterpret_cast<uint32_t*>(p + L.off_base);
  *keys_out = keys[0];
  *vals_out = vals[0];
  if (n <= 0) return hipSuccess;
  const int64_t tiles = plan.blocks;
  const int64_t nchunks = ceil_div(tiles, kChunk);
  const dim3 grid((unsigned)tiles), block(kSortBlock);
  hipError_t e;
  int cur = 0;
  for (int pass = 0; pass < plan.passes; ++pass) {
    const int shift = 8 * pass;
    const int bits = (plan.key_bits - shift) < 8 ? (plan.key_bits - shift) : 8;
    const int out = pass == 0 ? 0 : 1 - cur;
    const void* kin = pass == 0 ? (const void*)ids : (const void*)keys[cur];
    if (pass == 0)
      hipLaunchKernelGGL(sort_tile_hist_kernel<true>, grid, block, 0, stream, kin, n, shift, bits, R, hist, err);
    else
      hipLaunchKernelGGL(sort_tile_hist_kernel<false>, grid, block, 0, stream, kin, n, shift, bits, R, hist, err);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sort_chunk_sum_kernel, dim3((unsigned)nchunks), block, 0, stream,
                       (const uint32_t*)hist, tiles, chunk);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sort_chunk_scan_kernel, dim3(1), block, 0, stream, chunk, nchunks, base);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sort_chunk_apply_kernel, dim3((unsigned)nchunks), block, 0, stream, hist, tiles,
                       (const uint32_t*)chunk, (const uint32_t*)base);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (pass == 0)
      hipLaunchKernelGGL(sort_scatter_kernel<true>, grid, block, 0, stream, kin, (const uint32_t*)nullptr,
                         keys[out], vals[out], n, shift, bits, R, (const uint32_t*)hist);
    else
      hipLaunchKernelGGL(sort_scatter_kernel<false>, grid, block, 0, stream, kin, (const uint32_t*)vals[cur],
                         keys[out], vals[out], n, shift, bits, R, (const uint32_t*)hist);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    cur = out;
  }
  *keys_out = keys[cur];
  *vals_out = vals[cur];
  return hipSuccess;
}

}  // namespace gba
