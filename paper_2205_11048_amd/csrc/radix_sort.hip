// Stable LSD radix sort of the occurrence IDs, keyed by ID, carrying the
// occurrence index.  It groups the occurrences of each embedding ID so the
// push-step can deduplicate them and reduce their rows (Alg. 2: gradients of
// the embedding parameters are processed by ID).
//
// Each digit takes three launches: digit counts per chunk of four tiles, and
// per tile the counts of the earlier tiles of its chunk (1 KB per tile,
// tile-major); an exclusive scan of every digit's chunk counts, one block per
// digit; and a scatter in which each tile adds up its own offsets (digit
// start + chunk prefix + the tiles before it in its chunk), ranks its keys
// stably in LDS and writes runs of equal digits together.
// Ranks inside a wave come from ballots that match lanes holding the same
// digit, so skewed (Zipf) keys cost no LDS atomics on hot bins in the scatter.
#include "gba_device.hpp"
#include "gba_internal.hpp"

namespace gba {

constexpr int kSortBlock = 256;
constexpr int kSortWaves = kSortBlock / kWave;
// Keys per lane in the scatter: 16 (4096-key tiles) on the 8-bit passes, whose
// writes need long runs of equal digits; 8 (2048-key tiles) on the first,
// narrow-digit pass, where runs are long anyway and more resident blocks hide
// the latency of the 8-byte ID loads better.
constexpr int kItemsFirst = 8;
constexpr int kItemsRest = 16;
template <int ITEMS>
constexpr int64_t tile_keys() { return (int64_t)kSortBlock * ITEMS; }
constexpr int kRadix = 256;
constexpr int kXcds = 8;   // MI355X: 8 accelerator dies, each with its own L2
constexpr int kChunk = kSortWaves;                     // tiles per chunk: one hist block

__host__ __device__ static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

struct SortLayout {
  size_t arr, off_keys0, off_keys1, off_vals0, off_vals1, off_hist, off_chunk, off_total, bytes;
};

// tiles: the largest tile count of any pass (the first pass's)
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
  L.off_chunk = o; o += align_up((size_t)ceil_div((int64_t)nt, kChunk) * kRadix * 4);   // [chunk][digit]
  L.off_total = o; o += align_up(kRadix * 4);
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
// The check is a select, not a branch, so a lane's loads are all issued
// before the first one is waited for.
template <bool FIRST>
__device__ __forceinline__ uint32_t load_key(const void* src, int64_t i, int64_t R, bool* bad) {
  if (FIRST) {
    const int64_t id = static_cast<const int64_t*>(src)[i];
    const bool out = id < 0 || id >= R;
    *bad |= out;
    return out ? 0u : (uint32_t)id;
  }
  return static_cast<const uint32_t*>(src)[i];
}

// Digit counts of one tile into the wave's LDS row h_row.  Lane l holds keys
// tile0 + 4 * (l + 64 * c) + e, c < ITEMS, e < 4: each vector load of the
// wave covers 1 KB of consecutive keys.  FULL (every key of the tile exists)
// drops the bounds checks, so no branch waits on a load and a phase's loads
// are in flight together; only the last tile of a pass can be partial.
// Returns whether an ID outside [0, R) was seen (first pass).
template <bool FIRST, int ITEMS, bool FULL>
__device__ __forceinline__ bool count_tile(const void* __restrict__ keys_in, int64_t n, int64_t tile0, int shift,
                                           uint32_t mask, int64_t R, uint32_t* h_row, int lane) {
  constexpr int kHistKeys = 4 * ITEMS;   // keys per lane
  // eight vectors (32 keys) per lane per phase, all in flight together
  constexpr int kVecs = 8;
  static_assert(kHistKeys % (4 * kVecs) == 0, "whole phases per tile");
  bool bad = false;
#pragma unroll
  for (int ph = 0; ph < kHistKeys / 4 / kVecs; ++ph) {
    uint32_t digit[4 * kVecs];
#pragma unroll
    for (int cc = 0; cc < kVecs; ++cc) {
      const int c = ph * kVecs + cc;
      const int64_t i0 = tile0 + 4 * ((int64_t)lane + (int64_t)kWave * c);
      if (FULL || i0 + 3 < n) {
        uint32_t k4[4];
        if (FIRST) {
          const int64_t* ids = static_cast<const int64_t*>(keys_in);
          typedef int64_t i64x2 __attribute__((ext_vector_type(2)));
          const i64x2 a = *reinterpret_cast<const i64x2*>(ids + i0);
          const i64x2 b = *reinterpret_cast<const i64x2*>(ids + i0 + 2);
          const int64_t v[4] = {a.x, a.y, b.x, b.y};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool out = v[e] < 0 || v[e] >= R;
            bad |= out;
            k4[e] = out ? 0u : (uint32_t)v[e];
          }
        } else {
          const u32x4 v = *reinterpret_cast<const u32x4*>(static_cast<const uint32_t*>(keys_in) + i0);
          k4[0] = v.x; k4[1] = v.y; k4[2] = v.z; k4[3] = v.w;
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) digit[4 * cc + e] = (k4[e] >> shift) & mask;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          digit[4 * cc + e] = (i0 + e < n) ? (load_key<FIRST>(keys_in, i0 + e, R, &bad) >> shift) & mask : 0u;
      }
    }
    // one LDS add per run of equal digits among each lane's 4 consecutive keys
#pragma unroll
    for (int cc = 0; cc < kVecs; ++cc) {
      const int c = ph * kVecs + cc;
      const int64_t i0 = tile0 + 4 * ((int64_t)lane + (int64_t)kWave * c);
      uint32_t cur = digit[4 * cc];
      uint32_t len = (FULL || i0 < n) ? 1u : 0u;
#pragma unroll
      for (int e = 1; e < 4; ++e) {
        if (FULL || i0 + e < n) {
          if (digit[4 * cc + e] == cur) {
            ++len;
          } else {
            atomicAdd(&h_row[cur], len);
            cur = digit[4 * cc + e];
            len = 1;
          }
        }
      }
      if (len) atomicAdd(&h_row[cur], len);
    }
  }
  return bad;
}

// Digit counts of the four tiles of one chunk, one wave per tile; each adds
// one count per run of equal digits among each lane's 4 consecutive keys.
template <bool FIRST, int ITEMS>
__global__ void __launch_bounds__(kSortBlock)
sort_tile_hist_kernel(const void* __restrict__ keys_in, int64_t n, int64_t tiles, int shift, int bits,
                      int64_t R, uint32_t* __restrict__ hist, uint32_t* __restrict__ chunk,
                      int32_t* __restrict__ err) {
  __shared__ uint32_t h[kSortWaves][kRadix];
  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  for (int i = lane; i < kRadix; i += kWave) h[w][i] = 0u;
  __builtin_amdgcn_wave_barrier();
  const int64_t tile = (int64_t)blockIdx.x * kSortWaves + w;
  bool bad = false;
  if (tile < tiles) {
    const uint32_t mask = (1u << bits) - 1u;
    const int64_t tile0 = tile * tile_keys<ITEMS>();
    if (tile0 + tile_keys<ITEMS>() <= n)
      bad = count_tile<FIRST, ITEMS, true>(keys_in, n, tile0, shift, mask, R, h[w], lane);
    else
      bad = count_tile<FIRST, ITEMS, false>(keys_in, n, tile0, shift, mask, R, h[w], lane);
  }
  __syncthreads();
  // the block's tiles form one chunk: each tile's row holds the counts of the
  // chunk's earlier tiles (so the scatter needs one row, not a loop over
  // rows), and the chunk row holds the chunk's counts
  {
    const int d = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * kSortWaves;
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      if (t0 + k < tiles) hist[(t0 + k) * kRadix + d] = s;
      s += h[k][d];
    }
    chunk[(int64_t)blockIdx.x * kRadix + d] = s;
  }
  if (FIRST && bad) raise_error(err, GBA_DERR_ID_RANGE);
}

// One block per digit value: exclusive prefix of the digit's chunk counts, in
// place, and the digit's total.  Blocks of one XCD (block b runs on XCD b % 8)
// take 32 consecutive digits, so each 128-byte line of a chunk row is read by
// one XCD only.
constexpr int kDigitScanBatch = 8;
__global__ void __launch_bounds__(kSortBlock)
sort_digit_scan_kernel(uint32_t* __restrict__ chunk, int64_t nchunks, uint32_t* __restrict__ total) {
  __shared__ uint32_t tmp[kSortBlock / kWave + 1];
  const int d = (int)(blockIdx.x % kXcds) * (kRadix / kXcds) + (int)(blockIdx.x / kXcds);
  const int64_t per = ceil_div(nchunks, kSortBlock);
  const int64_t c_lo = (int64_t)threadIdx.x * per;
  const int64_t c_hi = (c_lo + per < nchunks) ? c_lo + per : nchunks;
  uint32_t s = 0;
  for (int64_t c0 = c_lo; c0 < c_hi; c0 += kDigitScanBatch) {
    uint32_t v[kDigitScanBatch];
#pragma unroll
    for (int k = 0; k < kDigitScanBatch; ++k) v[k] = (c0 + k < c_hi) ? chunk[(c0 + k) * kRadix + d] : 0u;
#pragma unroll
    for (int k = 0; k < kDigitScanBatch; ++k) s += v[k];
  }
  uint32_t all;
  uint32_t run = block_exclusive_scan<kSortBlock>(s, tmp, &all);
  for (int64_t c0 = c_lo; c0 < c_hi; c0 += kDigitScanBatch) {
    uint32_t v[kDigitScanBatch];
#pragma unroll
    for (int k = 0; k < kDigitScanBatch; ++k) v[k] = (c0 + k < c_hi) ? chunk[(c0 + k) * kRadix + d] : 0u;
#pragma unroll
    for (int k = 0; k < kDigitScanBatch; ++k) {
      if (c0 + k < c_hi) chunk[(c0 + k) * kRadix + d] = run;
      run += v[k];
    }
  }
  if (threadIdx.x == 0) total[d] = all;
}

// Tile of scatter block b.  Blocks are dispatched round-robin over the 8 XCDs
// (block b on XCD b % 8); giving XCD x the x-th eighth of the tiles, in order,
// puts neighbouring tiles on one L2, which then merges their partial-line
// writes into the same digit bucket before they reach HBM.
__device__ __forceinline__ int64_t xcd_tile(int64_t b, int64_t tiles) {
  const int64_t x = b % kXcds, i = b / kXcds, q = tiles / kXcds, r = tiles % kXcds;
  return x * q + (x < r ? x : r) + i;
}

// Exclusive scans of x and of y over the block, behind one barrier: every
// thread adds up the totals of the waves before its own.  `tmp` holds
// 2 * kSortWaves words.
__device__ __forceinline__ void block_exclusive_scan2(uint32_t x, uint32_t y, uint32_t* tmp, uint32_t* ex_x,
                                                      uint32_t* ex_y) {
  const int w = threadIdx.x / kWave;
  const uint32_t ix = wave_inclusive_scan(x), iy = wave_inclusive_scan(y);
  if (lane_id() == kWave - 1) {
    tmp[w] = ix;
    tmp[kSortWaves + w] = iy;
  }
  __syncthreads();
  uint32_t bx = 0, by = 0;
#pragma unroll
  for (int k = 0; k < kSortWaves; ++k) {
    if (k < w) {
      bx += tmp[k];
      by += tmp[kSortWaves + k];
    }
  }
  *ex_x = bx + ix - x;
  *ex_y = by + iy - y;
}

template <bool FIRST, int ITEMS>
__global__ void __launch_bounds__(kSortBlock)
sort_scatter_kernel(const void* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
                    uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out, int64_t n,
                    int shift, int bits, int64_t R, const uint32_t* __restrict__ hist,
                    const uint32_t* __restrict__ chunk, const uint32_t* __restrict__ total) {
  // per (wave, digit): the wave's count, then the tile position of the wave's
  // first key of that digit
  __shared__ uint32_t cnt[kSortWaves][kRadix];
  // per digit: the output position minus the tile position of its keys
  // (first the chunk and tile offset alone), and the digit total
  __shared__ uint32_t gshift[kRadix];
  __shared__ uint32_t s_tot[kRadix];
  __shared__ uint32_t tmp[2 * kSortWaves];
  constexpr int64_t kTile = tile_keys<ITEMS>();
  __shared__ uint32_t s_keys[kTile];
  __shared__ uint32_t s_vals[kTile];
  const int64_t tile = xcd_tile(blockIdx.x, gridDim.x);   // the grid has one block per tile
  // Where the tile's keys of digit d go: where the digit starts (scan of the
  // digit totals), plus its count in earlier chunks, plus in earlier tiles of
  // this tile's chunk.  The loads are issued with the keys' and used only
  // after the ranking, where one scan finds both the digit starts and the
  // tile's own digit offsets.
  const int d = threadIdx.x;
  const uint32_t off = chunk[(tile / kChunk) * kRadix + d] + hist[tile * kRadix + d];
  const uint32_t tot = total[d];
  const int w = threadIdx.x / kWave;
  const int64_t tile0 = tile * kTile;
  const int64_t base = tile0 + (int64_t)w * (kWave * ITEMS) + lane_id();
  const uint32_t mask = (1u << bits) - 1u;
  const uint64_t lt = lanemask_lt();

  uint32_t key[ITEMS], val[ITEMS], rank[ITEMS];
  // Every lane loads (lanes past the end re-read the last key, n > 0), so no
  // branch waits on a load and all of a lane's loads are in flight at once.
  // An ID outside [0, R) is sorted as 0 (the histogram launch reports it);
  // the first pass's values are the positions themselves, formed when stored.
  {
    uint64_t raw[FIRST ? ITEMS : 1];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
      const int64_t i = base + (int64_t)r * kWave;
      const int64_t ic = i < n ? i : n - 1;
      if (FIRST) {
        raw[r] = static_cast<const uint64_t*>(keys_in)[ic];
      } else {
        key[r] = static_cast<const uint32_t*>(keys_in)[ic];
        val[r] = vals_in[ic];
      }
    }
    if (FIRST) {
#pragma unroll
      for (int r = 0; r < ITEMS; ++r) key[r] = raw[r] < (uint64_t)R ? (uint32_t)raw[r] : 0u;
    }
  }
  // parked in LDS during the ranking (registers are what limit residency)
  gshift[d] = off;
  s_tot[d] = tot;
  // each wave counts in its own row
  for (int i = lane_id(); i < kRadix; i += kWave) cnt[w][i] = 0u;
  __builtin_amdgcn_wave_barrier();
  // Stable rank within (wave, digit): rounds in index order, lanes in order.
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
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
    // thread d alone reads and rewrites column d of cnt and entry d of gshift
    uint32_t c[kSortWaves];
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      c[k] = cnt[k][d];
      s += c[k];
    }
    uint32_t ex, start;
    block_exclusive_scan2(s, s_tot[d], tmp, &ex, &start);
    gshift[d] = start + gshift[d] - ex;   // modulo 2^32
    uint32_t run = ex;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      cnt[k][d] = run;
      run += c[k];
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const int64_t i = base + (int64_t)r * kWave;
    if (i < n) {
      const uint32_t digit = (key[r] >> shift) & mask;
      const uint32_t pos = cnt[w][digit] + rank[r];
      s_keys[pos] = key[r];
      s_vals[pos] = FIRST ? (uint32_t)i : val[r];
    }
  }
  __syncthreads();
  const int64_t tile_n = (n - tile0) < kTile ? (n - tile0) : kTile;
  for (int i = threadIdx.x; i < tile_n; i += kSortBlock) {
    const uint32_t k = s_keys[i];
    const uint32_t g = gshift[(k >> shift) & mask] + (uint32_t)i;
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
  p.blocks = n > 0 ? ceil_div(n, tile_keys<kItemsFirst>()) : 0;
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
  uint32_t* total = reinterpret_cast<uint32_t*>(p + L.off_total);
  *keys_out = keys[0];
  *vals_out = vals[0];
  if (n <= 0) return hipSuccess;
  hipError_t e;
  int cur = 0;
  // the narrowest digit goes first: the first pass sees keys in arrival order,
  // and fewer bins there mean longer runs of equal digits to write
  const int first_bits = plan.key_bits - 8 * (plan.passes - 1);
  for (int pass = 0; pass < plan.passes; ++pass) {
    const int shift = pass == 0 ? 0 : first_bits + 8 * (pass - 1);
    const int bits = pass == 0 ? first_bits : 8;
    const int out = pass == 0 ? 0 : 1 - cur;
    const void* kin = pass == 0 ? (const void*)ids : (const void*)keys[cur];
    const int64_t tiles = ceil_div(n, pass == 0 ? tile_keys<kItemsFirst>() : tile_keys<kItemsRest>());
    const int64_t nchunks = ceil_div(tiles, kChunk);
    const dim3 grid((unsigned)tiles), block(kSortBlock);
    if (pass == 0)
      hipLaunchKernelGGL((sort_tile_hist_kernel<true, kItemsFirst>), dim3((unsigned)nchunks), block, 0, stream,
                         kin, n, tiles, shift, bits, R, hist, chunk, err);
    else
      hipLaunchKernelGGL((sort_tile_hist_kernel<false, kItemsRest>), dim3((unsigned)nchunks), block, 0, stream,
                         kin, n, tiles, shift, bits, R, hist, chunk, err);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sort_digit_scan_kernel, dim3(kRadix), block, 0, stream, chunk, nchunks, total);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (pass == 0)
      hipLaunchKernelGGL((sort_scatter_kernel<true, kItemsFirst>), grid, block, 0, stream, kin,
                         (const uint32_t*)nullptr, keys[out], vals[out], n, shift, bits, R, (const uint32_t*)hist,
                         (const uint32_t*)chunk, (const uint32_t*)total);
    else
      hipLaunchKernelGGL((sort_scatter_kernel<false, kItemsRest>), grid, block, 0, stream, kin,
                         (const uint32_t*)vals[cur], keys[out], vals[out], n, shift, bits, R,
                         (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    cur = out;
  }
  *keys_out = keys[cur];
  *vals_out = vals[cur];
  return hipSuccess;
}

}  // namespace gba
