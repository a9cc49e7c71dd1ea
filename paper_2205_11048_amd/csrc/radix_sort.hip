// Stable LSD radix sort of the occurrence IDs, keyed by ID, carrying the
// occurrence index.  It groups the occurrences of each embedding ID so the
// push-step can deduplicate them and reduce their rows (Alg. 2: gradients of
// the embedding parameters are processed by ID).
//
// Each pass over one digit (<= 8 bits) is three launches: a per-tile digit
// histogram, a device-wide exclusive scan of the histograms (digit-major, so
// the scan yields each tile's global offset per digit), and a scatter that
// ranks the tile stably in LDS before writing runs of equal digits together.
// Ranks inside a wave come from ballots that match lanes holding the same
// digit, so skewed (Zipf) keys cost no LDS atomics on hot bins.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kSortBlock = 256;
constexpr int kSortWaves = kSortBlock / kWave;
constexpr int kSortItems = 16;                        // per lane
constexpr int kSortWaveTile = kWave * kSortItems;      // 1024 keys per wave
constexpr int64_t kSortTile = kSortBlock * kSortItems; // 4096 keys per block
constexpr int kRadix = 256;

static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

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

template <bool FIRST>
__global__ void __launch_bounds__(kSortBlock)
sort_histogram_kernel(const void* __restrict__ keys_in, int64_t n, int shift, int bits, int64_t R,
                      int64_t num_tiles, uint32_t* __restrict__ hist, int32_t* __restrict__ err) {
  __shared__ uint32_t cnt[kSortWaves][kRadix];
  for (int i = threadIdx.x; i < kSortWaves * kRadix; i += kSortBlock) (&cnt[0][0])[i] = 0;
  __syncthreads();
  const int w = threadIdx.x / kWave;
  const int64_t base = (int64_t)blockIdx.x * kSortTile + (int64_t)w * kSortWaveTile + lane_id();
  const uint32_t mask = (1u << bits) - 1u;
  bool bad = false;
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t i = base + (int64_t)r * kWave;
    const bool active = i < n;
    const uint32_t key = active ? load_key<FIRST>(keys_in, i, R, &bad) : 0u;
    const uint32_t digit = (key >> shift) & mask;
    const uint64_t m = match_digit(digit, bits, active);
    if (active && (m & lanemask_lt()) == 0) cnt[w][digit] += (uint32_t)__popcll(m);
  }
  if (FIRST && bad) raise_error(err, GBA_DERR_ID_RANGE);
  __syncthreads();
  const int d = threadIdx.x;   // kSortBlock == kRadix
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kSortWaves; ++k) s += cnt[k][d];
  hist[(int64_t)d * num_tiles + blockIdx.x] = s;
}

template <bool FIRST>
__global__ void __launch_bounds__(kSortBlock)
sort_scatter_kernel(const void* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
                    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t n,
                    int shift, int bits, int64_t R, int64_t num_tiles,
                    const uint32_t* __restrict__ offsets) {
  __shared__ uint32_t cnt[kSortWaves][kRadix];
  __shared__ uint32_t digit_start[kRadix];
  __shared__ uint32_t global_base[kRadix];
  __shared__ uint32_t tmp[kSortBlock / kWave + 1];
  __shared__ uint32_t s_keys[kSortTile];
  __shared__ uint32_t s_vals[kSortTile];
  for (int i = threadIdx.x; i < kSortWaves * kRadix; i += kSortBlock) (&cnt[0][0])[i] = 0;
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
    global_base[d] = offsets[(int64_t)d * num_tiles + blockIdx.x];
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
    if ((int64_t)g < n) {   // always true when the histograms are consistent
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
  const size_t arr = align_up((size_t)(n > 0 ? n : 1) * sizeof(uint32_t));
  const size_t hist_words = (size_t)kRadix * (size_t)(p.blocks > 0 ? p.blocks : 1);
  p.bytes = 4 * arr + align_up(hist_words * sizeof(uint32_t)) +
            align_up(scan_workspace_bytes((int64_t)hist_words));
  return p;
}

hipError_t launch_sort_ids(const int64_t* ids, int64_t n, int64_t R, const SortPlan& plan, void* ws,
                           const uint32_t** keys_out, const uint32_t** vals_out, int32_t* err,
                           hipStream_t stream) {
  char* p = static_cast<char*>(ws);
  const size_t arr = align_up((size_t)(n > 0 ? n : 1) * sizeof(uint32_t));
  uint32_t* keys[2] = {reinterpret_cast<uint32_t*>(p), reinterpret_cast<uint32_t*>(p + arr)};
  uint32_t* vals[2] = {reinterpret_cast<uint32_t*>(p + 2 * arr), reinterpret_cast<uint32_t*>(p + 3 * arr)};
  const size_t hist_words = (size_t)kRadix * (size_t)(plan.blocks > 0 ? plan.blocks : 1);
  uint32_t* hist = reinterpret_cast<uint32_t*>(p + 4 * arr);
  void* scan_ws = p + 4 * arr + align_up(hist_words * sizeof(uint32_t));
  *keys_out = keys[0];
  *vals_out = vals[0];
  if (n <= 0) return hipSuccess;
  const dim3 grid((unsigned)plan.blocks), block(kSortBlock);
  int cur = 0;
  for (int pass = 0; pass < plan.passes; ++pass) {
    const int shift = 8 * pass;
    const int bits = (plan.key_bits - shift) < 8 ? (plan.key_bits - shift) : 8;
    const int out = pass == 0 ? 0 : 1 - cur;
    if (pass == 0) {
      hipLaunchKernelGGL(sort_histogram_kernel<true>, grid, block, 0, stream, (const void*)ids, n,
                         shift, bits, R, plan.blocks, hist, err);
    } else {
      hipLaunchKernelGGL(sort_histogram_kernel<false>, grid, block, 0, stream,
                         (const void*)keys[cur], n, shift, bits, R, plan.blocks, hist, err);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_exclusive_scan_u32(hist, hist, (int64_t)kRadix * plan.blocks, nullptr, scan_ws, stream);
    if (e != hipSuccess) return e;
    if (pass == 0) {
      hipLaunchKernelGGL(sort_scatter_kernel<true>, grid, block, 0, stream, (const void*)ids,
                         (const uint32_t*)nullptr, keys[out], vals[out], n, shift, bits, R,
                         plan.blocks, (const uint32_t*)hist);
    } else {
      hipLaunchKernelGGL(sort_scatter_kernel<false>, grid, block, 0, stream, (const void*)keys[cur],
                         (const uint32_t*)vals[cur], keys[out], vals[out], n, shift, bits, R,
                         plan.blocks, (const uint32_t*)hist);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    cur = out;
  }
  *keys_out = keys[cur];
  *vals_out = vals[cur];
  return hipSuccess;
}

}  // namespace gba
