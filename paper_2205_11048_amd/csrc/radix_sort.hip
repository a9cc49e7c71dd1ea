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
//
// Hot keys.  Embedding IDs are Zipf-skewed (the paper's Insight 2: a few IDs
// appear in most batches), so a few hundred IDs can hold half of all
// occurrences.  With the hot-key plan, one block first picks the IDs that are
// frequent in an evenly spaced sample of the input.  The first pass gives
// each of them a bin of its own next to the cold digit bins, counts the cold
// keys that fall between consecutive hot IDs, and writes every hot occurrence
// straight to its final position: the cold keys below it, plus the hot
// occurrences of smaller hot IDs, plus its stable rank in its bin.  The later
// passes sort only the cold keys, and the last one leaves a gap for the hot
// runs below each key.  The result is the same stable sort, element for
// element; which IDs are hot changes only the time it takes.
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
constexpr int kItemsHotFirst = 8;   // the first pass of the hot-key plan
// Below this many keys the plain plan keeps 2048-key tiles on every pass: the
// later passes then have twice the blocks (at 256 K keys, 125 instead of 63
// for 256 compute units), where long write runs matter less than filling the chip.
constexpr int64_t kNarrowTilesBelow = int64_t(1) << 20;
template <int ITEMS>
constexpr int64_t tile_keys() { return (int64_t)kSortBlock * ITEMS; }
constexpr int kRadix = 256;
constexpr int kXcds = 8;   // MI355X: 8 accelerator dies, each with its own L2
// Tiles per chunk (one hist block): one per wave, or four per wave where a
// pass has tiles enough (the digit scans then read a quarter of the chunk
// rows, while small passes keep their hist blocks spread over the chip).
constexpr int kChunk = kSortWaves;                       // the smallest chunk
constexpr int64_t kWideChunkTiles = 8192;                // tiles from which a pass takes 4 per wave
static int hist_tiles_per_wave(int64_t tiles) { return tiles >= kWideChunkTiles ? 4 : 1; }

// Hot-key plan.
constexpr int kHotSample = 16384;      // sampled positions (one block sorts them in LDS)
constexpr int kHotBlock = 1024;
constexpr int kHotCap = 254;           // most hot IDs (one bin each; the lookup reads one entry past H)
constexpr int kHotBuckets = 1024;      // lookup buckets over the top 10 key bits
constexpr uint32_t kHotMinCount = 4;   // a sampled ID must occur this often to be hot
constexpr int64_t kHotMinKeys = int64_t(1) << 22;   // below this the plain sort is used

// Pass kinds.
enum : int {
  kPlain = 0,      // n keys from the launch arguments
  kHotFirst = 1,   // first pass with hot bins: cold keys to the work arrays, hot ones to the final arrays
  kCold = 2,       // a middle pass over the cold keys (their count read on the device)
  kColdLast = 3    // the last pass over the cold keys, into the final arrays, past the hot runs
};

__host__ __device__ static inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
static inline size_t align_up(size_t x) { return (x + 255) & ~size_t(255); }

// Device tables of the hot-key plan (inside the workspace).
struct HotTables {
  uint32_t* ids;        // [256] hot IDs, ascending (the first H are used)
  uint16_t* bucket;     // [kHotBuckets] hot IDs whose top bits are below the bucket index
  uint32_t* prefix;     // [256] hot occurrences of the hot IDs before hot ID h ([H]: all of them)
  uint32_t* meta;       // [0] H, [1] number of cold keys
  uint32_t* iv_chunk;   // [chunks][256] cold keys per chunk by the number of hot IDs below them
  uint32_t* iv_total;   // [256] the same over all chunks
  uint8_t* digit;       // [n] first-pass digit of every key (written by the histogram launch)
  int bshift;           // key >> bshift is the key's bucket
  int split;            // hot occurrences go to their own array, grouped by hot ID (not among the cold keys)
};

struct SortLayout {
  size_t arr, off_keys0, off_keys1, off_vals0, off_vals1, off_keys2, off_vals2, off_hist, off_chunk, off_total,
      off_iv, off_iv_total, off_hot, off_digit, bytes;
};

// tiles: the largest tile count of any pass (the first pass's)
static SortLayout sort_layout(int64_t n, int64_t tiles, bool hot) {
  SortLayout L{};
  L.arr = align_up((size_t)(n > 0 ? n : 1) * sizeof(uint32_t));
  const size_t nt = (size_t)(tiles > 0 ? tiles : 1);
  const size_t chunk_bytes = align_up((size_t)ceil_div((int64_t)nt, kChunk) * kRadix * 4);
  size_t o = 0;
  L.off_keys0 = o; o += L.arr;
  L.off_keys1 = o; o += L.arr;
  L.off_vals0 = o; o += L.arr;
  L.off_vals1 = o; o += L.arr;
  L.off_hist = o;  o += align_up(nt * kRadix * 4);                       // [tile][digit]
  L.off_chunk = o; o += chunk_bytes;                                     // [chunk][digit]
  L.off_total = o; o += align_up(kRadix * 4);
  if (hot) {
    L.off_keys2 = o; o += L.arr;
    L.off_vals2 = o; o += L.arr;
    L.off_iv = o;    o += chunk_bytes;                                   // [chunk][hot IDs below]
    L.off_iv_total = o; o += align_up(kRadix * 4);
    L.off_hot = o;   o += 4096 + 256;                                    // ids, bucket, prefix, meta
    L.off_digit = o; o += align_up((size_t)(n > 0 ? n : 1) + 64);       // + a vector's overrun
  }
  L.bytes = o;
  return L;
}

static HotTables hot_tables(char* ws, const SortLayout& L, int key_bits) {
  HotTables t;
  char* h = ws + L.off_hot;
  t.ids = reinterpret_cast<uint32_t*>(h);              // 1 KB
  t.bucket = reinterpret_cast<uint16_t*>(h + 1024);    // 2 KB
  t.prefix = reinterpret_cast<uint32_t*>(h + 3072);    // 1 KB
  t.meta = reinterpret_cast<uint32_t*>(h + 4096);
  t.iv_chunk = reinterpret_cast<uint32_t*>(ws + L.off_iv);
  t.iv_total = reinterpret_cast<uint32_t*>(ws + L.off_iv_total);
  t.digit = reinterpret_cast<uint8_t*>(ws + L.off_digit);
  t.bshift = key_bits > 10 ? key_bits - 10 : 0;
  return t;
}

// Mask of the active lanes whose digit equals this lane's digit.  Per bit,
// the lanes that differ from this one are the ballot of the bit, flipped
// where this lane's bit is 1: ballot ^ (0 or all ones), OR-ed into a mask of
// mismatches (one sign-extending bit extract, a compare for the ballot and
// one three-input bit operation per 32-lane half).
__device__ __forceinline__ uint64_t match_digit(uint32_t digit, int bits, bool active) {
  uint32_t diff_lo, diff_hi;
  {
    const uint64_t on = __ballot(active);
    diff_lo = ~(uint32_t)on;
    diff_hi = ~(uint32_t)(on >> 32);
  }
  for (int b = 0; b < bits; ++b) {
    const uint32_t x = (uint32_t)((int32_t)(digit << (31 - b)) >> 31);   // 0 or all ones: the lane's bit b
    const uint64_t bal = __ballot(x != 0u);
    // diff | (ballot ^ x) in one gfx950 three-input bit operation (table: S0 | (S1 ^ S2))
    diff_lo = __builtin_amdgcn_bitop3_b32(diff_lo, (uint32_t)bal, x, 0xF6);
    diff_hi = __builtin_amdgcn_bitop3_b32(diff_hi, (uint32_t)(bal >> 32), x, 0xF6);
  }
  const uint64_t m = ~(((uint64_t)diff_hi << 32) | diff_lo);
  return active ? m : 0ull;
}

// The same match for a digit width known at compile time (the loop unrolled).
template <int BITS>
__device__ __forceinline__ uint64_t match_digit_n(uint32_t digit, bool active) {
  uint32_t diff_lo, diff_hi;
  {
    const uint64_t on = __ballot(active);
    diff_lo = ~(uint32_t)on;
    diff_hi = ~(uint32_t)(on >> 32);
  }
#pragma unroll
  for (int b = 0; b < BITS; ++b) {
    const uint32_t x = (uint32_t)((int32_t)(digit << (31 - b)) >> 31);
    const uint64_t bal = __ballot(x != 0u);
    diff_lo = __builtin_amdgcn_bitop3_b32(diff_lo, (uint32_t)bal, x, 0xF6);
    diff_hi = __builtin_amdgcn_bitop3_b32(diff_hi, (uint32_t)(bal >> 32), x, 0xF6);
  }
  const uint64_t m = ~(((uint64_t)diff_hi << 32) | diff_lo);
  return active ? m : 0ull;
}

// A copy of x that the compiler cannot tie to earlier uses of x, so values
// derived from it (LDS addresses) are recomputed where needed instead of
// being held in registers across a phase.
__device__ __forceinline__ uint32_t opaque(uint32_t x) {
  asm volatile("" : "+v"(x));
  return x;
}

// Number of hot IDs below `key`, and whether `key` is one of them.  The bucket
// table narrows the search to the hot IDs that share the key's top bits: up
// to two are compared without a branch (no loop, so the lookups of a lane's
// keys overlap); a crowded bucket (hot IDs that are close in value, such as
// rows numbered in order of first appearance) is searched by halving.
struct HotLookup {
  const uint16_t* bucket;   // LDS [kHotBuckets]
  const uint32_t* ids;      // LDS [>= H + 1]
  uint32_t H;
  int bshift;
  __device__ __forceinline__ uint32_t rank(uint32_t key, bool* hot) const {
    const uint32_t t = key >> bshift;
    const uint32_t lo = bucket[t];
    const uint32_t hi = t + 1 < (uint32_t)kHotBuckets ? (uint32_t)bucket[t + 1] : H;
    const uint32_t a0 = ids[lo], a1 = ids[lo + 1];   // lo + 1 <= H <= kHotCap: inside the table
    const bool in0 = lo < hi, in1 = lo + 1 < hi;
    uint32_t r = lo + ((in0 && a0 < key) ? 1u : 0u) + ((in1 && a1 < key) ? 1u : 0u);
    bool h = (in0 && a0 == key) || (in1 && a1 == key);
    if (hi > lo + 2) {   // three or more hot IDs in the bucket
      uint32_t l = lo, u = hi;
      while (l < u) {
        const uint32_t mid = (l + u) >> 1;
        if (ids[mid] < key) l = mid + 1;
        else u = mid;
      }
      r = l;
      h = l < hi && ids[l] == key;
    }
    *hot = h;
    return r;
  }
};

// Copies the hot tables into LDS (every thread of the block takes part; the
// caller puts a barrier after).
__device__ __forceinline__ void load_hot_tables(const HotTables& t, uint16_t* s_bucket, uint32_t* s_ids) {
  const uint32_t* b32 = reinterpret_cast<const uint32_t*>(t.bucket);
  uint32_t* s32 = reinterpret_cast<uint32_t*>(s_bucket);
  for (int i = threadIdx.x; i < kHotBuckets / 2; i += blockDim.x) s32[i] = b32[i];
  for (int i = threadIdx.x; i < 256; i += blockDim.x) s_ids[i] = t.ids[i];
}

// Picks the hot IDs: counts the IDs of kHotSample / 64 evenly spaced runs of
// 64 consecutive positions (one coalesced load per wave; single scattered
// positions would each cost a page walk) in an LDS hash table, keeps those seen at least kHotMinCount times (raising
// the bar until at most `cap` remain), sorts them and builds the bucket
// table.  Only the first kHotInsertRounds rounds insert new IDs; the
// later ones only count IDs already in the table (an ID frequent enough to
// matter is there by then), which keeps the table sparse and the probes
// short.  A sampled ID that finds no free slot within kHotProbe steps is not
// counted; the choice of hot IDs changes only the speed of the sort.
constexpr int kHotTable = 16384;   // slots (a power of two)
constexpr int kHotProbe = 64;
constexpr int kHotInsertRounds = 4;   // of kHotSample / kHotBlock
__global__ void __launch_bounds__(kHotBlock)
hot_select_kernel(const int64_t* __restrict__ ids, int64_t n, int64_t R, int cap, HotTables t) {
  __shared__ uint32_t s_key[kHotTable];
  __shared__ uint32_t s_cnt[kHotTable];
  __shared__ uint32_t s_tmp[kHotBlock / kWave + 1];
  __shared__ uint32_t s_list[256];
  __shared__ uint32_t s_hot[256];
  __shared__ uint32_t s_nlist;
  const int tid = threadIdx.x;
  constexpr uint32_t kNone = 0xffffffffu;   // not a valid key (keys are below 2^31 here)
  constexpr int kPer = kHotSample / kHotBlock;
  constexpr int kRuns = kHotSample / kWave;
  const int lane = lane_id();
  uint32_t smp[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    const int run = tid / kWave + e * (kHotBlock / kWave);   // wave w takes runs w, w + 16, ...
    int64_t p0 = ((2 * (int64_t)run + 1) * n) / (2 * (int64_t)kRuns) - kWave / 2;
    p0 = p0 < n - kWave ? p0 : n - kWave;
    p0 = p0 > 0 ? p0 : 0;
    int64_t p = p0 + lane;
    p = p < n ? p : n - 1;
    const int64_t id = ids[p];
    smp[e] = (id >= 0 && id < R) ? (uint32_t)id : kNone;
  }
  for (int i = tid; i < kHotTable; i += kHotBlock) {
    s_key[i] = kNone;
    s_cnt[i] = 0u;
  }
  if (tid == 0) s_nlist = 0u;
  __syncthreads();
#pragma unroll
  for (int e = 0; e < kPer; ++e) {
    if (e == kHotInsertRounds) __syncthreads();   // every insertion is done
    const uint32_t k = smp[e];
    if (k == kNone) continue;
    uint32_t h = (k * 2654435761u) >> (32 - 14);   // Fibonacci hashing onto 2^14 slots
    for (int probe = 0; probe < kHotProbe; ++probe) {
      uint32_t cur = s_key[h];
      if (cur == kNone) {
        if (e >= kHotInsertRounds) break;   // not in the table: not counted
        cur = atomicCAS(&s_key[h], kNone, k);
      }
      if (cur == kNone || cur == k) {
        atomicAdd(&s_cnt[h], 1u);
        break;
      }
      h = (h + 1) & (kHotTable - 1);
    }
  }
  static_assert(kHotTable == 1 << 14, "hash width");
  __syncthreads();
  uint32_t T = kHotMinCount;
  for (;;) {
    uint32_t c = 0;
    for (int i = tid; i < kHotTable; i += kHotBlock) c += s_cnt[i] >= T ? 1u : 0u;
    uint32_t tot;
    (void)block_exclusive_scan<kHotBlock>(c, s_tmp, &tot);
    if (tot <= (uint32_t)cap) break;
    T += 1 + T / 8;
  }
  for (int i = tid; i < kHotTable; i += kHotBlock)
    if (s_cnt[i] >= T) s_list[atomicAdd(&s_nlist, 1u)] = s_key[i];
  __syncthreads();
  const uint32_t H = s_nlist;
  if ((uint32_t)tid < H) {
    // rank among the chosen IDs (distinct), so they come out ascending
    const uint32_t k = s_list[tid];
    uint32_t r = 0;
    for (uint32_t j = 0; j < H; ++j) r += s_list[j] < k ? 1u : 0u;
    s_hot[r] = k;
  }
  __syncthreads();
  const int bshift = t.bshift;
  for (int b = tid; b < kHotBuckets; b += kHotBlock) {
    // hot IDs whose top bits are below b: the first index with id >= b << bshift
    const uint32_t lim = (uint32_t)b << bshift;
    uint32_t lo = 0, hi = H;
    while (lo < hi) {
      const uint32_t mid = (lo + hi) >> 1;
      if (s_hot[mid] < lim) lo = mid + 1;
      else hi = mid;
    }
    t.bucket[b] = (uint16_t)lo;
  }
  if (tid < 256) t.ids[tid] = (uint32_t)tid < H ? s_hot[tid] : kNone;
  if (tid == 0) t.meta[0] = H;
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

// Digit of a key on a hot-key first pass: a hot ID's own bin past the cold
// bins, else its low bits.  Cold keys are also counted by the hot IDs below
// them (iv, LDS).
__device__ __forceinline__ uint32_t hot_first_digit(uint32_t key, uint32_t mask, uint32_t cold_bins,
                                                    const HotLookup& hl, bool* hot, uint32_t* below) {
  *below = hl.rank(key, hot);
  return *hot ? cold_bins + *below : (key & mask);
}

// Copies of each digit counter in a histogram row, interleaved (lane l adds
// to copy l % kHistCopies, in the next LDS bank): lanes that add to the same
// frequent digit (a hot ID) touch different words.
constexpr int kHistCopies = 4;

// Digit counts of one tile into the wave's LDS row h_row.  Lane l holds keys
// tile0 + 4 * (l + 64 * c) + e, c < ITEMS, e < 4: each vector load of the
// wave covers 1 KB of consecutive keys.  FULL (every key of the tile exists)
// drops the bounds checks, so no branch waits on a load and a phase's loads
// are in flight together; only the last tile of a pass can be partial.
// Returns whether an ID outside [0, R) was seen (first pass).
template <bool FIRST, int ITEMS, bool FULL, bool HOT, bool IV>
__device__ __forceinline__ bool count_tile(const void* __restrict__ keys_in, int64_t n, int64_t tile0, int shift,
                                           uint32_t mask, int64_t R, uint32_t* h_row, int lane,
                                           const HotLookup& hl, uint32_t cold_bins, uint32_t* iv,
                                           uint8_t* __restrict__ dig_out) {
  constexpr int kHistKeys = 4 * ITEMS;   // keys per lane
  // eight vectors (32 keys) per lane per phase, all in flight together; on
  // the first pass, whose 8-byte IDs take twice the registers, four (two with
  // the hot lookup), which keeps the kernel at 8 waves per SIMD
  constexpr int kVecs = HOT ? 2 : (FIRST ? 4 : 8);
  static_assert(kHistKeys % (4 * kVecs) == 0, "whole phases per tile");
  bool bad = false;
#pragma unroll
  for (int ph = 0; ph < kHistKeys / 4 / kVecs; ++ph) {
    uint32_t digit[4 * kVecs];
#pragma unroll
    for (int cc = 0; cc < kVecs; ++cc) {
      const int c = ph * kVecs + cc;
      const int64_t i0 = tile0 + 4 * ((int64_t)lane + (int64_t)kWave * c);
      uint32_t k4[4];
      if (FULL || i0 + 3 < n) {
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
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) k4[e] = (i0 + e < n) ? load_key<FIRST>(keys_in, i0 + e, R, &bad) : 0u;
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (HOT) {
          bool hot;
          uint32_t below;
          digit[4 * cc + e] = hot_first_digit(k4[e], mask, cold_bins, hl, &hot, &below);
          if (IV && !hot && (FULL || i0 + e < n)) atomicAdd(&iv[below], 1u);
        } else {
          digit[4 * cc + e] = (k4[e] >> shift) & mask;
        }
      }
      if (HOT) {   // the scatter reads the digits instead of looking the keys up again
        if (FULL || i0 + 3 < n) {
          *reinterpret_cast<uint32_t*>(dig_out + i0) = digit[4 * cc] | (digit[4 * cc + 1] << 8) |
                                                        (digit[4 * cc + 2] << 16) | (digit[4 * cc + 3] << 24);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (i0 + e < n) dig_out[i0 + e] = (uint8_t)digit[4 * cc + e];
        }
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
            atomicAdd(&h_row[cur * kHistCopies + (lane % kHistCopies)], len);
            cur = digit[4 * cc + e];
            len = 1;
          }
        }
      }
      if (len) atomicAdd(&h_row[cur * kHistCopies + (lane % kHistCopies)], len);
    }
  }
  return bad;
}

// Digit counts of the tiles of one chunk (4 or 16), one wave per tile; each
// adds one count per run of equal digits among each lane's 4 consecutive keys.
// kCold reads the key count from n_dev; kHotFirst also writes the chunk's
// counts of cold keys by the number of hot IDs below them.
// Eight waves per SIMD: the blocks of a pass are then all resident at once
// where the grid allows (at 65.5 M keys the hot-key first pass has 2000
// blocks of 16 waves; the cold passes have some 500 active blocks).
template <bool FIRST, int ITEMS, int MODE, int TPW>
__global__ void __launch_bounds__(kSortWaves * TPW * kWave) __attribute__((amdgpu_waves_per_eu(8, 8)))
sort_tile_hist_kernel(const void* __restrict__ keys_in, int64_t n_arg, const uint32_t* __restrict__ n_dev,
                      int shift, int bits, int64_t R, uint32_t* __restrict__ hist, uint32_t* __restrict__ chunk,
                      HotTables ht, int32_t* __restrict__ err) {
  constexpr bool HOT = MODE == kHotFirst;
  constexpr int kTiles = kSortWaves * TPW;   // the chunk: one tile per wave
  static_assert(kTiles * kWave >= kRadix, "a thread per digit for the chunk rows");
  __shared__ uint32_t h[kTiles][kRadix * kHistCopies];
  __shared__ uint32_t s_bucket_w[HOT ? kHotBuckets / 2 : 1];   // uint16 entries
  __shared__ uint32_t s_ids[HOT ? 256 : 1];
  __shared__ uint32_t s_iv[HOT ? kRadix : 1];
  uint16_t* s_bucket = reinterpret_cast<uint16_t*>(s_bucket_w);
  const int64_t n = MODE == kCold ? (int64_t)*n_dev : n_arg;
  const int64_t tiles = ceil_div(n, tile_keys<ITEMS>());
  const int w = threadIdx.x / kWave;
  const int lane = lane_id();
  for (int i = lane; i < kRadix * kHistCopies; i += kWave) h[w][i] = 0u;
  HotLookup hl{s_bucket, s_ids, 0u, ht.bshift};
  uint32_t cold_bins = 0;
  if (HOT) {
    load_hot_tables(ht, s_bucket, s_ids);
    if (threadIdx.x < kRadix) s_iv[threadIdx.x] = 0u;
    hl.H = ht.meta[0];
    cold_bins = 1u << bits;
    __syncthreads();
  } else {
    __builtin_amdgcn_wave_barrier();
  }
  // wave w counts the chunk's tile w into row w
  bool bad = false;
  const int64_t tile = (int64_t)blockIdx.x * kTiles + w;
  if (tile < tiles) {
    const uint32_t mask = (1u << bits) - 1u;
    const int64_t tile0 = tile * tile_keys<ITEMS>();
    // the cold keys' counts by hot IDs below them are needed only for the
    // merged output (split: the segment pass finds them from the sorted keys)
    const bool full = tile0 + tile_keys<ITEMS>() <= n;
    if (HOT && !ht.split) {
      if (full)
        bad |= count_tile<FIRST, ITEMS, true, HOT, true>(keys_in, n, tile0, shift, mask, R, h[w], lane, hl, cold_bins,
                                                         s_iv, ht.digit);
      else
        bad |= count_tile<FIRST, ITEMS, false, HOT, true>(keys_in, n, tile0, shift, mask, R, h[w], lane, hl,
                                                          cold_bins, s_iv, ht.digit);
    } else {
      if (full)
        bad |= count_tile<FIRST, ITEMS, true, HOT, false>(keys_in, n, tile0, shift, mask, R, h[w], lane, hl,
                                                          cold_bins, s_iv, ht.digit);
      else
        bad |= count_tile<FIRST, ITEMS, false, HOT, false>(keys_in, n, tile0, shift, mask, R, h[w], lane, hl,
                                                           cold_bins, s_iv, ht.digit);
    }
  }
  __syncthreads();
  // the block's tiles form one chunk: each tile's row holds the counts of the
  // chunk's earlier tiles (so the scatter needs one row, not a loop over
  // rows), and the chunk row holds the chunk's counts
  if (threadIdx.x < kRadix) {
    const int d = threadIdx.x;
    const int64_t t0 = (int64_t)blockIdx.x * kTiles;
    uint32_t s = 0;
#pragma unroll
    for (int k = 0; k < kTiles; ++k) {
      if (t0 + k < tiles) hist[(t0 + k) * kRadix + d] = s;
      uint32_t c = 0;
#pragma unroll
      for (int j = 0; j < kHistCopies; ++j) c += h[k][d * kHistCopies + j];
      s += c;
    }
    chunk[(int64_t)blockIdx.x * kRadix + d] = s;
    if (HOT && !ht.split) ht.iv_chunk[(int64_t)blockIdx.x * kRadix + d] = s_iv[d];
  }
  if (FIRST && bad) raise_error(err, GBA_DERR_ID_RANGE);
}

// One block per digit value: exclusive prefix of the digit's chunk counts, in
// place, and the digit's total.  Blocks of one XCD (block b runs on XCD b % 8)
// take 32 consecutive digits, so each 128-byte line of a chunk row is read by
// one XCD only.  With a second array (iv), blocks kRadix.. add up its columns
// into iv_total (no prefix).
constexpr int kDigitScanBatch = 8;
__global__ void __launch_bounds__(kSortBlock)
sort_digit_scan_kernel(uint32_t* __restrict__ chunk, int64_t nchunks, uint32_t* __restrict__ total,
                       const uint32_t* __restrict__ iv, uint32_t* __restrict__ iv_total) {
  __shared__ uint32_t tmp[kSortBlock / kWave + 1];
  const bool second = blockIdx.x >= kRadix;
  const int b = second ? blockIdx.x - kRadix : blockIdx.x;
  const int d = (int)(b % kXcds) * (kRadix / kXcds) + (int)(b / kXcds);
  const uint32_t* src = second ? iv : chunk;
  const int64_t per = ceil_div(nchunks, kSortBlock);
  const int64_t c_lo = (int64_t)threadIdx.x * per;
  const int64_t c_hi = (c_lo + per < nchunks) ? c_lo + per : nchunks;
  uint32_t s = 0;
  for (int64_t c0 = c_lo; c0 < c_hi; c0 += kDigitScanBatch) {
    uint32_t v[kDigitScanBatch];
#pragma unroll
    for (int k = 0; k < kDigitScanBatch; ++k) v[k] = (c0 + k < c_hi) ? src[(c0 + k) * kRadix + d] : 0u;
#pragma unroll
    for (int k = 0; k < kDigitScanBatch; ++k) s += v[k];
  }
  uint32_t all;
  uint32_t run = block_exclusive_scan<kSortBlock>(s, tmp, &all);
  if (second) {
    if (threadIdx.x == 0) iv_total[d] = all;
    return;
  }
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

// Tile of scatter block b with the tiles handed to the XCDs in chunks of C
// consecutive tiles (chunk c on XCD c % 8), for the 8-bit passes: all XCDs
// write inside one window of each digit's output (fewer, denser write
// streams than one eighth of the tiles per XCD), and the neighbouring tiles
// of a chunk still share an L2.  Tiles past the last whole round of 8 C
// chunks keep their own index; a pass with fewer tiles than one round uses
// the eighths.
constexpr int kXcdChunk = 64;
template <int C>
__device__ __forceinline__ int64_t xcd_chunk_tile(int64_t b, int64_t tiles) {
  const int64_t round = (int64_t)kXcds * C;
  if (tiles < round) return xcd_tile(b, tiles);
  if (b >= (tiles / round) * round) return b;   // the tail, in order
  const int64_t x = b % kXcds, i = b / kXcds;
  return ((i / C) * kXcds + x) * C + i % C;
}

// Exclusive scans of V values over the block, behind one barrier: every
// thread adds up the totals of the waves before its own.  `tmp` holds
// V * kSortWaves words.
template <int V>
__device__ __forceinline__ void block_exclusive_scan_v(const uint32_t (&x)[V], uint32_t* tmp, uint32_t (&ex)[V],
                                                       uint32_t (&all)[V]) {
  const int w = threadIdx.x / kWave;
  uint32_t inc[V];
#pragma unroll
  for (int v = 0; v < V; ++v) inc[v] = wave_inclusive_scan(x[v]);
  if (lane_id() == kWave - 1) {
#pragma unroll
    for (int v = 0; v < V; ++v) tmp[v * kSortWaves + w] = inc[v];
  }
  __syncthreads();
#pragma unroll
  for (int v = 0; v < V; ++v) {
    uint32_t b = 0, t = 0;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      const uint32_t u = tmp[v * kSortWaves + k];
      if (k < w) b += u;
      t += u;
    }
    ex[v] = b + inc[v] - x[v];
    all[v] = t;
  }
}

// Scatter of one tile.  kHotFirst writes cold keys to keys_out/vals_out and
// hot ones to their final places in keys_fin/vals_fin (split: grouped by hot
// ID, from 0, with no cold keys between them); kColdLast writes the
// cold keys to keys_out/vals_out (the final arrays), each past the hot runs of
// the hot IDs below it.  n_total bounds the final arrays.
// Every pass but the hot-key first stages its keys and then its values through
// one LDS buffer (a key's output place follows from the key, and is kept in a
// register for its value), so a block needs 22 KB of LDS instead of 38 KB;
// the hot-key first pass, whose digits travel beside the keys, stages both.
template <bool FIRST, int ITEMS, int MODE>
__device__ __forceinline__ void
scatter_tile(const void* __restrict__ keys_in, const uint32_t* __restrict__ vals_in,
             uint32_t* __restrict__ keys_out, uint32_t* __restrict__ vals_out,
             uint32_t* __restrict__ keys_fin, uint32_t* __restrict__ vals_fin, int64_t n_arg,
             const uint32_t* __restrict__ n_dev, int64_t n_total, int shift, int bits, int64_t R,
             const uint32_t* __restrict__ hist, const uint32_t* __restrict__ chunk,
             const uint32_t* __restrict__ total, const HotTables& ht, int chunk_shift) {
  constexpr bool HOT = MODE == kHotFirst;
  constexpr bool DYN = MODE == kCold || MODE == kColdLast;
  constexpr bool GAP = MODE == kColdLast;
  constexpr bool ONE_BUF = !HOT;
  // per (wave, digit): the wave's count, then the tile position of the wave's
  // first key of that digit (kColdLast: then the hot tables)
  __shared__ uint32_t cnt[kSortWaves][kRadix];
  // per digit: the output position minus the tile position of its keys
  // (first the chunk and tile offset alone), and the digit total
  __shared__ uint32_t gshift[kRadix];
  __shared__ uint32_t s_tot[kRadix];
  __shared__ uint32_t tmp[4 * kSortWaves];
  constexpr int kTile = (int)tile_keys<ITEMS>();
  __shared__ uint32_t s_keys[kTile];
  __shared__ uint32_t s_vals[ONE_BUF ? 1 : kTile];
  const int64_t n = DYN ? (int64_t)*n_dev : n_arg;
  const int64_t tiles = DYN ? ceil_div(n, kTile) : (int64_t)gridDim.x;
  if (DYN && (int64_t)blockIdx.x >= tiles) return;   // the grid is sized for every key
  const int64_t tile = HOT ? xcd_tile(blockIdx.x, tiles) : xcd_chunk_tile<kXcdChunk>(blockIdx.x, tiles);
  // Where the tile's keys of digit d go: where the digit starts (scan of the
  // digit totals), plus its count in earlier chunks, plus in earlier tiles of
  // this tile's chunk.  The loads are issued with the keys' and used only
  // after the ranking, where one scan finds both the digit starts and the
  // tile's own digit offsets.
  const int d = threadIdx.x;
  const uint32_t off = chunk[(tile >> chunk_shift) * kRadix + d] + hist[tile * kRadix + d];
  const uint32_t tot = total[d];
  // hot bin d (ID d - cold_bins) starts after the cold keys with at most
  // d - cold_bins hot IDs below them: thread d takes column d - cold_bins
  uint32_t iv_tot = 0;
  if (HOT && !ht.split && d >= (1 << bits)) iv_tot = ht.iv_total[d - (1 << bits)];
  // kColdLast: this thread's share of the hot tables, parked in registers
  // until the ranking is done with cnt
  uint32_t g_prefix = 0, g_id = 0, g_bucket0 = 0, g_bucket1 = 0, g_H = 0;
  if (GAP) {
    g_prefix = ht.prefix[d];
    g_id = ht.ids[d];
    const uint32_t* b32 = reinterpret_cast<const uint32_t*>(ht.bucket);
    g_bucket0 = b32[d];
    g_bucket1 = b32[d + kSortBlock];
    g_H = ht.meta[0];
  }
  const int w = threadIdx.x / kWave;
  const int64_t tile0 = tile * kTile;
  // keys in this tile (only the last tile of a pass is partial), and the tile
  // position of this lane's first key: indices inside a tile are 32-bit
  const int tile_n = (n - tile0) < kTile ? (int)(n - tile0) : kTile;
  const int lbase = w * (kWave * ITEMS) + lane_id();
  const uint32_t mask = (1u << bits) - 1u;
  const uint64_t lt = lanemask_lt();
  const int bshift = ht.bshift;

  uint32_t key[ITEMS], val[ITEMS], rank[ITEMS];
  // kHotFirst: each key's digit (8 bits, from the histogram launch), four to a register
  uint32_t dig_hot[HOT ? (ITEMS + 3) / 4 : 1] = {};
  // Every lane loads (lanes past the end re-read the last key, n > 0), so no
  // branch waits on a load and all of a lane's loads are in flight at once.
  // An ID outside [0, R) is sorted as 0 (the histogram launch reports it);
  // the first pass's values are the positions themselves, formed when stored.
  {
    uint64_t raw[FIRST ? ITEMS : 1];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
      const int li = lbase + r * kWave;
      const int64_t ic = tile0 + (li < tile_n ? li : tile_n - 1);
      if (FIRST) {
        raw[r] = static_cast<const uint64_t*>(keys_in)[ic];
        if (HOT) dig_hot[r / 4] |= (uint32_t)ht.digit[ic] << (8 * (r % 4));
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
  const uint32_t cold_bins = HOT ? (1u << bits) : 0u;
  uint32_t H = 0;
  if (HOT) H = ht.meta[0];
  __builtin_amdgcn_wave_barrier();
  auto dig = [&](int r) -> uint32_t {
    return HOT ? (dig_hot[r / 4] >> (8 * (r % 4))) & 0xffu : (key[r] >> shift) & mask;
  };
  auto active_at = [&](int r) -> bool { return lbase + r * kWave < tile_n; };
  // Stable rank within (wave, digit): rounds in index order, lanes in order.
  // Every pass but a plain first one has 8-bit digits (hot-key first: digit bytes).
  constexpr bool kBits8 = HOT || !FIRST;
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const bool active = active_at(r);
    const uint32_t digit = dig(r);
    const uint64_t m = kBits8 ? match_digit_n<8>(digit, active) : match_digit(digit, bits, active);
    uint32_t before = 0;
    if (active) before = cnt[w][digit];
    // every lane of the wave has read the counter before the leader updates it
    __builtin_amdgcn_wave_barrier();
    if (active && (m & lt) == 0) cnt[w][digit] = before + (uint32_t)__popcll(m);
    // (materialised here: a rank held as its 64-bit lane mask takes two registers)
    // (on the hot-key first pass the compiler's own placement is kept: at
    // more than 5 waves per SIMD that VALU-bound pass runs slower)
    rank[r] = HOT ? before + (uint32_t)__popcll(m & lt) : opaque(before + (uint32_t)__popcll(m & lt));
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
    if (HOT) {
      // cold bins start where the cold keys before them end; hot bin h starts
      // after every cold key below hot ID h (iv columns 0..h) and every hot
      // occurrence of the hot IDs before it
      const bool cold = (uint32_t)d < cold_bins;
      const uint32_t x[4] = {s, cold ? s_tot[d] : 0u, cold ? 0u : s_tot[d], iv_tot};
      uint32_t e4[4], a4[4];
      block_exclusive_scan_v<4>(x, tmp, e4, a4);
      ex = e4[0];
      start = cold ? e4[1] : (ht.split ? e4[2] : e4[2] + e4[3] + x[3]);
      if (blockIdx.x == 0) {
        // for the later passes: hot occurrences below each hot ID, cold keys
        if (!cold) ht.prefix[d - cold_bins] = e4[2];
        if (d == 0) {
          ht.prefix[H] = a4[2];
          ht.meta[1] = a4[1];
        }
      }
    } else {
      const uint32_t x[2] = {s, s_tot[d]};
      uint32_t e2[2], a2[2];
      block_exclusive_scan_v<2>(x, tmp, e2, a2);
      ex = e2[0];
      start = e2[1];
    }
    gshift[d] = start + gshift[d] - ex;   // modulo 2^32
    uint32_t run = ex;
#pragma unroll
    for (int k = 0; k < kSortWaves; ++k) {
      cnt[k][d] = run;
      run += c[k];
    }
  }
  __syncthreads();
  if (ONE_BUF) {
    // each key's tile position in digit order, then the keys staged
    // (the digit taken again from the key: the counter addresses of the
    // ranking are not held through the scan)
    uint32_t pos[ITEMS];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) pos[r] = cnt[w][(opaque(key[r]) >> shift) & mask] + rank[r];
#pragma unroll
    for (int r = 0; r < ITEMS; ++r)
      if (active_at(r)) s_keys[pos[r]] = key[r];
    __syncthreads();
    // staged position i = threadIdx.x + r * kSortBlock goes to out[r]
    uint32_t out[ITEMS];
    const int64_t bound = GAP ? n_total : n;   // always above out when the counts are consistent
    if (GAP) {
      // cnt is free now: the hot prefix [0, 256), hot IDs [256, 512), buckets [512, 1024)
      uint32_t* c32 = &cnt[0][0];
      c32[d] = g_prefix;
      c32[256 + d] = g_id;
      c32[512 + d] = g_bucket0;
      c32[512 + kSortBlock + d] = g_bucket1;
      __syncthreads();
      const HotLookup gl{reinterpret_cast<const uint16_t*>(c32 + 512), c32 + 256, g_H, bshift};
#pragma unroll
      for (int r = 0; r < ITEMS; ++r) {
        const int i = threadIdx.x + r * kSortBlock;
        out[r] = 0u;
        if (i < tile_n) {
          const uint32_t k = s_keys[i];
          bool hot;
          const uint32_t below = gl.rank(k, &hot);
          out[r] = gshift[(k >> shift) & mask] + (uint32_t)i + c32[below];
          if ((int64_t)out[r] < bound) keys_out[out[r]] = k;
        }
      }
    } else {
#pragma unroll
      for (int r = 0; r < ITEMS; ++r) {
        const int i = threadIdx.x + r * kSortBlock;
        out[r] = 0u;
        if (i < tile_n) {
          const uint32_t k = s_keys[i];
          out[r] = gshift[(k >> shift) & mask] + (uint32_t)i;
          if ((int64_t)out[r] < bound) keys_out[out[r]] = k;
        }
      }
    }
    __syncthreads();   // every key is read out before the values take the buffer
#pragma unroll
    for (int r = 0; r < ITEMS; ++r)
      if (active_at(r)) s_keys[pos[r]] = FIRST ? (uint32_t)(tile0 + lbase + r * kWave) : val[r];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < ITEMS; ++r) {
      const int i = threadIdx.x + r * kSortBlock;
      if (i < tile_n && (int64_t)out[r] < bound) vals_out[out[r]] = s_keys[i];
    }
    return;
  }
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    if (active_at(r)) {
      const int li = lbase + r * kWave;
      const uint32_t dr = dig(r);
      const uint32_t pos = cnt[w][dr] + rank[r];
      s_keys[pos] = key[r];
      // kHotFirst: the digit beside the key's place in the tile
      s_vals[pos] = (uint32_t)li | (dr << 16);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < tile_n; i += kSortBlock) {
    const uint32_t k = s_keys[i];
    const uint32_t v = s_vals[i];
    const uint32_t digit = v >> 16;
    const uint32_t val_out = (uint32_t)tile0 + (v & 0xffffu);
    const uint32_t g = gshift[digit] + (uint32_t)i;
    uint32_t* ko = keys_out;
    uint32_t* vo = vals_out;
    bool store_key = true;
    if (digit >= cold_bins) {   // a hot ID: straight to its final place
      ko = keys_fin;
      vo = vals_fin;
      store_key = !ht.split;    // split: only the occurrence indices are read
    }
    if ((int64_t)g < n) {   // always true when the counts are consistent
      if (store_key) ko[g] = k;
      vo[g] = val_out;
    }
  }
}

#define GBA_SCATTER_PARAMS                                                                              \
  const void* __restrict__ keys_in, const uint32_t* __restrict__ vals_in, uint32_t* __restrict__ keys_out,  \
      uint32_t* __restrict__ vals_out, uint32_t* __restrict__ keys_fin, uint32_t* __restrict__ vals_fin,   \
      int64_t n_arg, const uint32_t* __restrict__ n_dev, int64_t n_total, int shift, int bits, int64_t R,   \
      const uint32_t* __restrict__ hist, const uint32_t* __restrict__ chunk,                               \
      const uint32_t* __restrict__ total, HotTables ht, int chunk_shift
#define GBA_SCATTER_ARGS                                                                                         \
  keys_in, vals_in, keys_out, vals_out, keys_fin, vals_fin, n_arg, n_dev, n_total, shift, bits, R, hist, chunk, total, \
      ht, chunk_shift

template <bool FIRST, int ITEMS, int MODE>
__global__ void __launch_bounds__(kSortBlock) sort_scatter_kernel(GBA_SCATTER_PARAMS) {
  scatter_tile<FIRST, ITEMS, MODE>(GBA_SCATTER_ARGS);
}

// The hot-key first pass.
__global__ void __launch_bounds__(kSortBlock) sort_scatter_hot_first_kernel(GBA_SCATTER_PARAMS) {
  scatter_tile<true, kItemsHotFirst, kHotFirst>(GBA_SCATTER_ARGS);
}

SortPlan plan_sort(int64_t n, int64_t R, int hot_mode) {
  SortPlan p{};
  p.n = n;
  int bits = 1;
  while (bits < 32 && ((int64_t)1 << bits) < R) ++bits;
  p.key_bits = bits;
  p.passes = (bits + 7) / 8;
  p.first_bits = bits - 8 * (p.passes - 1);
  // The hot plan needs room for hot bins beside the first pass's cold bins; a
  // key whose width is a whole number of bytes gets a first pass of hot bins
  // only (one cold bin), which pays when it saves a full pass of cold keys.
  bool hot = bits >= 9 && bits <= 31 && n > 0;
  int hot_passes = p.passes, hot_first = p.first_bits;
  if (p.first_bits == 8) {
    hot_passes = p.passes + 1;
    hot_first = 0;
    hot = hot && p.passes >= 3;
  }
  if (hot_mode == 0) hot = false;
  if (hot_mode < 0) hot = hot && n >= kHotMinKeys;
  p.hot = hot;
  if (hot) {
    p.passes = hot_passes;
    p.first_bits = hot_first;
    const int cold_bins = 1 << hot_first;
    p.hot_cap = kRadix - cold_bins < kHotCap ? kRadix - cold_bins : kHotCap;
  }
  p.blocks = n > 0 ? ceil_div(n, tile_keys<kItemsFirst>()) : 0;
  p.bytes = sort_layout(n, p.blocks, p.hot).bytes;
  return p;
}

hipError_t launch_sort_ids(const int64_t* ids, int64_t n, int64_t R, const SortPlan& plan, void* ws,
                           const uint32_t** keys_out, const uint32_t** vals_out, int32_t* err,
                           hipStream_t stream, SortHot* split) {
  const SortLayout L = sort_layout(n, plan.blocks, plan.hot);
  char* p = static_cast<char*>(ws);
  uint32_t* keys[3] = {reinterpret_cast<uint32_t*>(p + L.off_keys0), reinterpret_cast<uint32_t*>(p + L.off_keys1),
                       plan.hot ? reinterpret_cast<uint32_t*>(p + L.off_keys2) : nullptr};
  uint32_t* vals[3] = {reinterpret_cast<uint32_t*>(p + L.off_vals0), reinterpret_cast<uint32_t*>(p + L.off_vals1),
                       plan.hot ? reinterpret_cast<uint32_t*>(p + L.off_vals2) : nullptr};
  uint32_t* hist = reinterpret_cast<uint32_t*>(p + L.off_hist);
  uint32_t* chunk = reinterpret_cast<uint32_t*>(p + L.off_chunk);
  uint32_t* total = reinterpret_cast<uint32_t*>(p + L.off_total);
  HotTables ht{};
  if (plan.hot) ht = hot_tables(p, L, plan.key_bits);
  ht.split = (plan.hot && split) ? 1 : 0;
  *keys_out = keys[plan.hot && !split ? 2 : 0];
  *vals_out = vals[plan.hot && !split ? 2 : 0];
  if (split) {
    *split = SortHot{};
    if (plan.hot) {
      split->n_cold = ht.meta + 1;
      split->hot_vals = vals[2];
      split->ids = ht.ids;
      split->bucket = ht.bucket;
      split->prefix = ht.prefix;
      split->meta = ht.meta;
      split->bshift = ht.bshift;
    }
  }
  if (n <= 0) return hipSuccess;
  hipError_t e;
  const dim3 block(kSortBlock);
  if (plan.hot) {
    hipLaunchKernelGGL(hot_select_kernel, dim3(1), dim3(kHotBlock), 0, stream, ids, n, R, plan.hot_cap, ht);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  int cur = 0;
  const bool narrow = !plan.hot && n < kNarrowTilesBelow;
  // the narrowest digit goes first: the first pass sees keys in arrival order,
  // and fewer bins there mean longer runs of equal digits to write
  const int first_bits = plan.first_bits;
  const uint32_t* n_cold = plan.hot ? ht.meta + 1 : nullptr;
  for (int pass = 0; pass < plan.passes; ++pass) {
    const int shift = pass == 0 ? 0 : first_bits + 8 * (pass - 1);
    const int bits = pass == 0 ? first_bits : 8;
    const bool last = pass == plan.passes - 1;
    const bool gap = plan.hot && last && !ht.split;   // merged output: the cold keys make room for the hot runs
    const int out = pass == 0 ? 0 : (gap ? 2 : 1 - cur);
    const void* kin = pass == 0 ? (const void*)ids : (const void*)keys[cur];
    const int64_t tiles =
        ceil_div(n, pass > 0 ? (narrow ? tile_keys<kItemsFirst>() : tile_keys<kItemsRest>())
                             : (plan.hot ? tile_keys<kItemsHotFirst>() : tile_keys<kItemsFirst>()));
    const int tpw = hist_tiles_per_wave(tiles);
    const int chunk_tiles = kSortWaves * tpw;
    const int chunk_shift = chunk_tiles == 16 ? 4 : 2;
    const int64_t nchunks = ceil_div(tiles, chunk_tiles);
    const dim3 grid((unsigned)tiles), hgrid((unsigned)nchunks);
#define GBA_HIST(F, IT, MD, NDEV)                                                                            \
  if (tpw == 4)                                                                                              \
    hipLaunchKernelGGL((sort_tile_hist_kernel<F, IT, MD, 4>), hgrid, dim3(4 * kSortWaves * kWave), 0, stream, kin, n, \
                       NDEV, shift, bits, R, hist, chunk, ht, err);                                          \
  else                                                                                                       \
    hipLaunchKernelGGL((sort_tile_hist_kernel<F, IT, MD, 1>), hgrid, dim3(kSortWaves * kWave), 0, stream, kin, n,     \
                       NDEV, shift, bits, R, hist, chunk, ht, err);
    static_assert(kSortWaves == 4, "chunk_shift assumes 4 or 16 tiles per chunk");
    if (pass == 0 && plan.hot) {
      GBA_HIST(true, kItemsHotFirst, kHotFirst, (const uint32_t*)nullptr)
    } else if (pass == 0) {
      GBA_HIST(true, kItemsFirst, kPlain, (const uint32_t*)nullptr)
    } else if (plan.hot) {
      GBA_HIST(false, kItemsRest, kCold, n_cold)
    } else if (narrow) {
      GBA_HIST(false, kItemsFirst, kPlain, (const uint32_t*)nullptr)
    } else {
      GBA_HIST(false, kItemsRest, kPlain, (const uint32_t*)nullptr)
    }
#undef GBA_HIST
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const bool with_iv = pass == 0 && plan.hot && !ht.split;
    hipLaunchKernelGGL(sort_digit_scan_kernel, dim3(with_iv ? 2 * kRadix : kRadix), block, 0, stream, chunk,
                       nchunks, total, (const uint32_t*)ht.iv_chunk, ht.iv_total);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const uint32_t* vin = pass == 0 ? (const uint32_t*)nullptr : (const uint32_t*)vals[cur];
    if (pass == 0 && plan.hot)
      hipLaunchKernelGGL(sort_scatter_hot_first_kernel, grid, block, 0, stream, kin, vin,
                         keys[0], vals[0], keys[2], vals[2], n, (const uint32_t*)nullptr, n, shift, bits, R,
                         (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total, ht, chunk_shift);
    else if (pass == 0)
      hipLaunchKernelGGL((sort_scatter_kernel<true, kItemsFirst, kPlain>), grid, block, 0, stream, kin, vin,
                         keys[0], vals[0], (uint32_t*)nullptr, (uint32_t*)nullptr, n, (const uint32_t*)nullptr, n,
                         shift, bits, R, (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total, ht,
                         chunk_shift);
    else if (gap)
      hipLaunchKernelGGL((sort_scatter_kernel<false, kItemsRest, kColdLast>), grid, block, 0, stream, kin, vin,
                         keys[out], vals[out], (uint32_t*)nullptr, (uint32_t*)nullptr, n, n_cold, n, shift, bits,
                         R, (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total, ht, chunk_shift);
    else if (plan.hot)
      hipLaunchKernelGGL((sort_scatter_kernel<false, kItemsRest, kCold>), grid, block, 0, stream, kin, vin,
                         keys[out], vals[out], (uint32_t*)nullptr, (uint32_t*)nullptr, n, n_cold, n, shift, bits,
                         R, (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total, ht, chunk_shift);
    else if (narrow)
      hipLaunchKernelGGL((sort_scatter_kernel<false, kItemsFirst, kPlain>), grid, block, 0, stream, kin, vin,
                         keys[out], vals[out], (uint32_t*)nullptr, (uint32_t*)nullptr, n, (const uint32_t*)nullptr,
                         n, shift, bits, R, (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total,
                         ht, chunk_shift);
    else
      hipLaunchKernelGGL((sort_scatter_kernel<false, kItemsRest, kPlain>), grid, block, 0, stream, kin, vin,
                         keys[out], vals[out], (uint32_t*)nullptr, (uint32_t*)nullptr, n, (const uint32_t*)nullptr,
                         n, shift, bits, R, (const uint32_t*)hist, (const uint32_t*)chunk, (const uint32_t*)total,
                         ht, chunk_shift);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    cur = out;
  }
  *keys_out = keys[cur];
  *vals_out = vals[cur];
  return hipSuccess;
}

}  // namespace gba
